// sf_kernels_vg.hip -- gfx950 kernels for the per-key-channel (vector) gate.
//
// With a gate g_t in R^{d_k} the recurrence is S_t = diag(a_t) S_{t-1} + k_t v_t^T,
// a_t = exp(g_t) (the GLA-style decay of Sec. 2.1 with one factor per key
// row), o_t = S_t^T q_t.  In the chunkwise form (Sec. 2.2) the cumulative
// log-decay b[t][c] = sum_{u<=t} g_u[c] (chunk-local, inclusive, base 2 here)
// is a matrix, so the intra-chunk scores carry the decay inside their channel
// contraction:
//   A[t][s] = sum_c q[t][c] k[s][c] 2^(b[t][c] - b[s][c])        (s <= t)
//   O       = (Q o 2^b) S + A V
//   S_next  = diag(2^b63) S + (K o 2^(b63 - b))^T V
// All the per-element factors are staged with the tiles: Q~ = Q o 2^b (<= 1)
// and K^ = K o 2^-b, so that A = Q~ K^^T is a plain MFMA product and
// (K o 2^(b63-b)) = diag(2^b63) K^, i.e. S_next = diag(2^b63) (S + K^^T V).
// K^ is bounded by 2^100 |k| when every channel decays by at most 2^-100 inside
// the chunk; a chunk that decays faster in some channel is walked token by
// token instead (exact recurrence, slower), decided per chunk and workgroup.
//
// Kernels (wave w of D/(16 NCT) waves owns NCT state column tiles: NCT = 2 for
// the preps and the dq walk, NCT = 1 for the o, dv and dk walks, whose state
// then fits in half the registers and two waves share each SIMD):
//   k_prep_vg<BWD=false>  D_J and the per-channel superchunk decay
//   k_prep_vg<BWD=true>   E_J = sum_t diag(2^{B_t}) q_t dO_t^T
//   k_prep_vg_bwd         the backward's replay of D_J and its E_J in one launch
//   k_walk_vg             o (and S_out for a one-superchunk segment)
//   k_dq_vg               dq and q o dq (into dg) by a forward walk
//   k_dv_vg               dv by a reverse walk with G
//   k_dk_vg               dk and dg by a reverse walk with G^T
// The superchunk scans are the scalar ones with per-row decay (k_scan<.., true>).
#include "sf_chunk.hpp"

namespace sf {

namespace {

constexpr float kMinChunkLog2 = -100.f;  // fast path iff every channel keeps >= 2^-100

// fp32 per-channel gate tile with the element ownership of Tile<T, D, NT>:
// thread tid holds rows row0 .. row0+RPT-1 of channels cb*E .. cb*E+E-1.
template <typename T, int D, int NT>
struct GTile {
    using TT = Tile<T, D, NT>;
    static constexpr int E = TT::E, RPT = TT::RPT, CB = TT::CB, NV = E / 4;
    static constexpr int SCR = NT / 64 * D;  // floats of gate_cumsum scratch
    f32x4 r[RPT][NV];
    __device__ __forceinline__ void load(const float *g, int64_t ls, int tid) {
        const float *p = g + (int64_t)(tid / CB) * RPT * ls + (tid % CB) * E;
#pragma unroll
        for (int j = 0; j < RPT; ++j)
#pragma unroll
            for (int v = 0; v < NV; ++v) r[j][v] = *reinterpret_cast<const f32x4 *>(p + (int64_t)j * ls + 4 * v);
    }
    __device__ __forceinline__ float at(int j, int c) const { return r[j][c >> 2][c & 3]; }
};

// Per-channel inclusive cumulative log2-decay over the chunk for this thread's
// tile elements (b[j][c]) and the chunk totals of its channels (tot[c]).
// A thread sums its own rows in registers; the row groups of a wave (threads
// CB lanes apart) are combined by lane swaps (DPP rotate within a 16-lane row,
// then the 16- and 32-lane swaps of gfx950), the waves through scratch
// (NT/64 x D floats).  Every thread adds the wave totals in the same order, so
// tot[c] is the same value in every thread, and it is also the value of the
// last row's b.  There is one barrier inside; the
// caller must pass a barrier before scratch is written again.
template <typename T, int D, int NT>
__device__ __forceinline__ void gate_cumsum(const GTile<T, D, NT> &gt, float (&b)[GTile<T, D, NT>::RPT][GTile<T, D, NT>::E],
                                            float (&tot)[GTile<T, D, NT>::E], float *scratch, int tid) {
    using G = GTile<T, D, NT>;
    constexpr int E = G::E, RPT = G::RPT, CB = G::CB, NW = NT / 64;
    static_assert(CB == 8 || CB == 16 || CB == 32, "row groups of a wave");
    const int lane = tid & 63, ch0 = (tid % CB) * E;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    float pre[E], wt[E];
#pragma unroll
    for (int c = 0; c < E; ++c) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            acc += gt.at(j, c) * LOG2E;
            b[j][c] = acc;
        }
        // exclusive prefix over the wave's lower row groups (p) and the wave total (x)
        float x = acc, p = 0.f;
        if constexpr (CB == 8) {  // the other group of the 16-lane row: lanes l ^ 8
            const float z = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x128, 0xf, 0xf, false));
            if (lane & 8) p = z;
            x += z;
        }
        if constexpr (CB <= 16) {  // rows 2r, 2r+1 of the wave: [0] the even row's, [1] the odd row's
            const unsigned u = __builtin_bit_cast(unsigned, x);
            const auto s = __builtin_amdgcn_permlane16_swap(u, u, false, false);
            const float lo = __builtin_bit_cast(float, (unsigned)s[0]), hi = __builtin_bit_cast(float, (unsigned)s[1]);
            if (lane & 16) p += lo;
            x = lo + hi;
        }
        {  // lanes 0-31 and 32-63: [0] the lower half's, [1] the upper half's
            const unsigned u = __builtin_bit_cast(unsigned, x);
            const auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
            const float lo = __builtin_bit_cast(float, (unsigned)s[0]), hi = __builtin_bit_cast(float, (unsigned)s[1]);
            if (lane & 32) p += lo;
            x = lo + hi;
        }
        pre[c] = p;
        wt[c] = x;
    }
    if (lane < CB) {
#pragma unroll
        for (int v = 0; v < G::NV; ++v)
            *reinterpret_cast<f32x4 *>(&scratch[w * D + ch0 + 4 * v]) = f32x4{wt[4 * v], wt[4 * v + 1], wt[4 * v + 2], wt[4 * v + 3]};
    }
    __syncthreads();
    float pw[E];
#pragma unroll
    for (int c = 0; c < E; ++c) pw[c] = 0.f;
    for (int v2 = 0; v2 < w; ++v2) {  // waves before this one
#pragma unroll
        for (int v = 0; v < G::NV; ++v) {
            const f32x4 x = *reinterpret_cast<const f32x4 *>(&scratch[v2 * D + ch0 + 4 * v]);
#pragma unroll
            for (int u = 0; u < 4; ++u) pw[4 * v + u] += x[u];
        }
    }
#pragma unroll
    for (int c = 0; c < E; ++c) tot[c] = pw[c];
    for (int v2 = w; v2 < NW; ++v2) {
#pragma unroll
        for (int v = 0; v < G::NV; ++v) {
            const f32x4 x = *reinterpret_cast<const f32x4 *>(&scratch[v2 * D + ch0 + 4 * v]);
#pragma unroll
            for (int u = 0; u < 4; ++u) tot[4 * v + u] += x[u];
        }
    }
#pragma unroll
    for (int j = 0; j < RPT; ++j)
#pragma unroll
        for (int c = 0; c < E; ++c) b[j][c] += pw[c] + pre[c];
    // the chunk's last row is its total, to the bit: factors 2^(tot - b) of that
    // row are exactly 1 however far the chunk decays (its exponent would
    // otherwise carry the rounding of a sum of magnitude |tot|)
    if (tid / CB == NT / CB - 1) {
#pragma unroll
        for (int c = 0; c < E; ++c) b[RPT - 1][c] = tot[c];
    }
}

// Stores tile t scaled per element by f[j][c] as a hi/lo pair of natural tiles:
// nat_pos channel order when NAT, else plain channel order with rows that have
// bit 3 set swizzled by swx.
template <typename T, int D, int NT, bool NAT>
__device__ __forceinline__ void store_scaled(const Tile<T, D, NT> &t, const float (&f)[Tile<T, D, NT>::RPT][Tile<T, D, NT>::E],
                                             T *hi, T *lo, int ld, int tid, int swx) {
    using TT = Tile<T, D, NT>;
    constexpr int E = TT::E;
    typedef T h4 __attribute__((ext_vector_type(4)));
    const int ch = t.cb(tid) * E, r0 = t.row0(tid);
#pragma unroll
    for (int j = 0; j < TT::RPT; ++j) {
        const int row = r0 + j;
#pragma unroll
        for (int u = 0; u < E / 4; ++u) {
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = tof<T>(t.r[j][4 * u + e]) * f[j][4 * u + e];
            h4 vh = {}, vl = {};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                vh[e] = cvt<T>(x[e]);
                vl[e] = cvt<T>(x[e] - tof<T>(vh[e]));
            }
            const int col = NAT ? nat_pos(ch + 4 * u) : ((ch + 4 * u) ^ (((row >> 3) & 1) * swx));
            *reinterpret_cast<h4 *>(hi + row * ld + col) = vh;
            if constexpr (kSplit<T>) *reinterpret_cast<h4 *>(lo + row * ld + col) = vl;
        }
    }
}

// a += x * y for hi/lo pairs, leaving out lo*lo (3 MFMAs)
template <typename T>
__device__ __forceinline__ void mma3(f32x4 &acc, const frag_t<T> &xh, const frag_t<T> &xl, const frag_t<T> &yh,
                                     const frag_t<T> &yl) {
    mma(acc, xh, yh);
    if constexpr (kSplit<T>) {
        mma(acc, xl, yh);
        mma(acc, xh, yl);
    }
}

template <typename T>
__device__ __forceinline__ f32x4 ld4(const T *p) {
    return ld4f(p);
}

}  // namespace

// ---------------------------------------------------------------------------
// Pre (vector gate): per superchunk
//   D_J = sum_c diag(decay after c) (K_c o 2^(b63 - b))^T V_c,  Lg_J[c] = log2 decay
//   E_J = sum_t diag(2^{B_t}) q_t dO_t^T  (BWD; B superchunk-local, inclusive)
// Every factor is <= 1; the scaled key (query) tile is the shared exact-split
// A operand, V (dO) the wave's own columns.
// One superchunk (item) of either summary; the LDS arrays are the caller's:
// sX, sXl (C x (D + pad) each), sY (the same), scratch (the gate cumsum's) and
// sE63 (D floats).
template <typename T, int D, int NCT, bool BWD>
__device__ __forceinline__ void prep_vg_item(const SegArgs &a, int item, T *sX, T *sXl, T *sY, float *scratch,
                                             float *sE63) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplit<T>;
    using TT = Tile<T, D, NT>;
    using GT = GTile<T, D, NT>;
    constexpr int E = TT::E, RPT = TT::RPT;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a, item);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *X = (const T *)(BWD ? a.q : a.k) + xo;
    const T *Y = (const T *)(BWD ? a.dO : a.v) + xo;
    const float *gp = a.g + d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const int grp = tid / TT::CB, ch0 = (tid % TT::CB) * E;

    f32x4 Acc[NCT][NK];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) Acc[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    float off[E];  // log2 decay of the superchunk's earlier chunks, this thread's channels
#pragma unroll
    for (int c = 0; c < E; ++c) off[c] = 0.f;

    TT tx, ty;
    GT tg;
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        tx.load(X + nx, a.sx_l, tid);
        ty.load(Y + nx, a.sx_l, tid);
        tg.load(gp + (int64_t)c * C * a.sg_l, a.sg_l, tid);
    };
    issue(0);

    for (int c = 0; c < d.nch; ++c) {
        __syncthreads();
        float b[RPT][E], tot[E], f[RPT][E];
        gate_cumsum<T, D, NT>(tg, b, tot, scratch, tid);
#pragma unroll
        for (int j = 0; j < RPT; ++j)
#pragma unroll
            for (int cc = 0; cc < E; ++cc) f[j][cc] = BWD ? fexp2(off[cc] + b[j][cc]) : fexp2(tot[cc] - b[j][cc]);
        store_scaled<T, D, NT, false>(tx, f, sX, sXl, LDN, tid, SWX);
        ty.store_swz(sY, LDN, tid, SWX);
        if (!BWD && grp == 0) {
#pragma unroll
            for (int cc = 0; cc < E; ++cc) sE63[ch0 + cc] = fexp2(tot[cc]);
        }
#pragma unroll
        for (int cc = 0; cc < E; ++cc) off[cc] += tot[cc];
        if (c + 1 < d.nch) issue(c + 1);
        __syncthreads();
        if constexpr (!BWD) {
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const f32x4 ev = *reinterpret_cast<const f32x4 *>(&sE63[16 * i + 4 * q4]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) Acc[ct][i] *= ev;
            }
        }
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> yf[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) yf[ct] = ldfragTR<T, LDN, SWX>(sY, tro, 32 * ks, 16 * (NCT * w + ct));
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> xh = ldfragTR<T, LDN, SWX>(sX, tro, 32 * ks, 16 * i);
                frag_t<T> xl = {};
                if constexpr (SP) xl = ldfragTR<T, LDN, SWX>(sXl, tro, 32 * ks, 16 * i);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    mma(Acc[ct][i], xh, yf[ct]);
                    if constexpr (SP) mma(Acc[ct][i], xl, yf[ct]);
                }
            }
        }
    }
    const int64_t so = ((int64_t)d.bh * a.n_super + d.J) * D * D;
    float *dst = BWD ? a.wsE : a.wsS;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dst[so + (int64_t)(16 * i + 4 * q4 + r) * D + 16 * (NCT * w + ct) + n16] = Acc[ct][i][r];
    if (!BWD && grp == 0) {
        float *lg = a.wsLg + ((int64_t)d.bh * a.n_super + d.J) * D;
#pragma unroll
        for (int cc = 0; cc < E; ++cc) lg[ch0 + cc] = off[cc];
    }
}

#define SF_PREP_VG_LDS                                                           \
    constexpr int LDN = D + pad<T>();                                          \
    __shared__ __attribute__((aligned(16))) T sX[C * LDN];                     \
    __shared__ __attribute__((aligned(16))) T sXl[kSplit<T> ? C * LDN : 8];    \
    __shared__ __attribute__((aligned(16))) T sY[C * LDN];                     \
    __shared__ __attribute__((aligned(16))) float scratch[GTile<T, D, 64 * D / (16 * NCT)>::SCR]; \
    __shared__ __attribute__((aligned(16))) float sE63[D];

template <typename T, int D, int NCT, bool BWD>
__global__ void __launch_bounds__(64 * D / (16 * NCT), sizeof(T) == 2 ? 2 : 1) k_prep_vg(SegArgs a) {
    SF_PREP_VG_LDS
    prep_vg_item<T, D, NCT, BWD>(a, (int)blockIdx.x, sX, sXl, sY, scratch, sE63);
}

// The backward's two summaries in one launch: workgroups [0, n) replay D_J,
// [n, 2n) form E_J (n = B H n_super); two workgroups share a CU, so the two
// halves overlap.
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), sizeof(T) == 2 ? 2 : 1) k_prep_vg_bwd(SegArgs a) {
    SF_PREP_VG_LDS
    const int n = (int)(gridDim.x / 2), item = (int)blockIdx.x;
    if (item < n) prep_vg_item<T, D, NCT, false>(a, item, sX, sXl, sY, scratch, sE63);
    else prep_vg_item<T, D, NCT, true>(a, item - n, sX, sXl, sY, scratch, sE63);
}
#undef SF_PREP_VG_LDS

// ---------------------------------------------------------------------------
// Forward walker (vector gate): o over the chunks of one superchunk.
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), 1) k_walk_vg(SegArgs a) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplit<T>;
    using TT = Tile<T, D, NT>;
    using GT = GTile<T, D, NT>;
    constexpr int E = TT::E, RPT = TT::RPT;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // Q o 2^b, nat_pos order (hi)
    __shared__ __attribute__((aligned(16))) T sQl[SP ? C * LDN : 8];
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];   // K o 2^-b, plain, swizzled (hi)
    __shared__ __attribute__((aligned(16))) T sKl[SP ? C * LDN : 8];
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];   // plain, swizzled
    constexpr int AB = 2 * C * LDT * (int)sizeof(T), SB = GT::SCR * 4;
    __shared__ __attribute__((aligned(16))) char sAraw[AB > SB ? AB : SB];  // A hi/lo, or the gate scratch
    T *sA = reinterpret_cast<T *>(sAraw), *sAl = sA + C * LDT;
    float *scratch = reinterpret_cast<float *>(sAraw);
    __shared__ __attribute__((aligned(16))) float sE63[D];
    __shared__ int sFast;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    T *Y = (T *)a.o + xo;
    const float *gp = a.g + d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const int64_t SS = (int64_t)D * D;
    const int grp = tid / TT::CB, ch0 = (tid % TT::CB) * E;

    const float *src = a.n_super == 1 ? (a.S_in ? a.S_in + d.bh * SS : nullptr)
                                      : a.wsS + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 S[NCT][NK];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int col = 16 * (NCT * w + ct) + n16, row = 16 * i + 4 * q4;
#pragma unroll
            for (int r = 0; r < 4; ++r) S[ct][i][r] = src ? src[(int64_t)(row + r) * D + col] : 0.f;
        }

    TT t1, t2, t3;
    GT tg;
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        t1.load(Q + nx, a.sx_l, tid);
        t2.load(K + nx, a.sx_l, tid);
        t3.load(V + nx, a.sx_l, tid);
        tg.load(gp + (int64_t)c * C * a.sg_l, a.sg_l, tid);
    };
    issue(0);

    for (int c = 0; c < d.nch; ++c) {
        __syncthreads();
        if (tid == 0) sFast = 1;
        float b[RPT][E], tot[E];
        gate_cumsum<T, D, NT>(tg, b, tot, scratch, tid);
        bool ok = true;
#pragma unroll
        for (int cc = 0; cc < E; ++cc) ok = ok && tot[cc] >= kMinChunkLog2;
        if (!ok) sFast = 0;
        {
            float f[RPT][E];
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = fexp2(b[j][cc]);
            store_scaled<T, D, NT, true>(t1, f, sQ, sQl, LDN, tid, SWX);
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = ok ? fexp2(-b[j][cc]) : 0.f;
            store_scaled<T, D, NT, false>(t2, f, sK, sKl, LDN, tid, SWX);
        }
        t3.store_swz(sV, LDN, tid, SWX);
        if (grp == 0) {
#pragma unroll
            for (int cc = 0; cc < E; ++cc) sE63[ch0 + cc] = fexp2(tot[cc]);
        }
        if (c + 1 < d.nch) issue(c + 1);
        __syncthreads();
        const bool fast = sFast != 0;
        __syncthreads();  // every wave has read the flag (and the scratch is free)

        if (fast) {
            // scores P^T[s][t] = sum_ch K^[s][ch] Q~[t][ch] on the causal tiles -> A[t][s]
            for (int i = w; i < 10; i += NW) {
                int tt, st;
                tri_tile(i, tt, st);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    const frag_t<T> kh = ldfrag_swz<T, LDN, SWX>(sK, swo, 16 * st, 32 * ks);
                    const frag_t<T> qh = ldfrag_unperm<T>(sQ, LDN, 16 * tt, 32 * ks, lane);
                    frag_t<T> kl = {}, ql = {};
                    if constexpr (SP) {
                        kl = ldfrag_swz<T, LDN, SWX>(sKl, swo, 16 * st, 32 * ks);
                        ql = ldfrag_unperm<T>(sQl, LDN, 16 * tt, 32 * ks, lane);
                    }
                    mma3<T>(p, kh, kl, qh, ql);
                }
                const int t = 16 * tt + n16;
                float v4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v4[r] = 16 * st + 4 * q4 + r <= t ? p[r] : 0.f;
                const int o = t * LDT + 16 * st + 4 * q4;
                st4_split<T>(&sA[o], &sAl[SP ? o : 0], v4);
            }
            // A tiles read by the A.V product but above the diagonal are zero
            for (int e = tid; e < 512; e += NT) {
                const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
                const int idx = tile ? (32 + rr) * LDT + 48 + cc : rr * LDT + 16 + cc;
                sA[idx] = cvt<T>(0.f);
                if constexpr (SP) sAl[idx] = cvt<T>(0.f);
            }
            __syncthreads();

            frag_t<T> vf[NCT][C / 32];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int c0 = 16 * (NCT * w + ct);
                f32x4 O[4];
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) O[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    frag_t<T> fh, fl;
                    split_acc<T>(S[ct][2 * ks], S[ct][2 * ks + 1], fh, fl);
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) {
                        frag_t<T> qh = ldfrag(sQ, LDN, 16 * tt, 32 * ks, lane), ql = {};
                        if constexpr (SP) ql = ldfrag(sQl, LDN, 16 * tt, 32 * ks, lane);
                        mma3<T>(O[tt], fh, fl, qh, ql);
                    }
                }
#pragma unroll
                for (int ks = 0; ks < C / 32; ++ks) {
                    vf[ct][ks] = ldfragTR<T, LDN, SWX>(sV, tro, 32 * ks, c0);
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) {
                        if (32 * ks > 16 * tt + 15) continue;
                        mma(O[tt], vf[ct][ks], ldfrag(sA, LDT, 16 * tt, 32 * ks, lane));
                        if constexpr (SP) mma(O[tt], vf[ct][ks], ldfrag(sAl, LDT, 16 * tt, 32 * ks, lane));
                    }
                }
#pragma unroll
                for (int tt = 0; tt < 4; ++tt)
                    st4(Y + (int64_t)(c * C + 16 * tt + n16) * a.sx_l + c0 + 4 * q4, O[tt][0], O[tt][1], O[tt][2],
                        O[tt][3]);
            }
            // S = diag(2^b63) (S + K^^T V)
#pragma unroll
            for (int ks = 0; ks < C / 32; ++ks)
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const frag_t<T> kh = ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, 16 * i);
                    frag_t<T> kl = {};
                    if constexpr (SP) kl = ldfragTR<T, LDN, SWX>(sKl, tro, 32 * ks, 16 * i);
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) mma2<T>(S[ct][i], kh, kl, vf[ct][ks]);
                }
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const f32x4 ev = *reinterpret_cast<const f32x4 *>(&sE63[16 * i + 4 * q4]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) S[ct][i] *= ev;
            }
        } else {
            // token by token: S = diag(a_t) S + k_t v_t^T, o_t = S^T q_t
            for (int t = 0; t < C; ++t) {
                const int64_t tok = (int64_t)c * C + t;
                float vv[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) vv[ct] = tof<T>(V[tok * a.sx_l + 16 * (NCT * w + ct) + n16]);
                float part[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) part[ct] = 0.f;
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const int row = 16 * i + 4 * q4;
                    const f32x4 gv = *reinterpret_cast<const f32x4 *>(gp + tok * a.sg_l + row);
                    const f32x4 kv = ld4<T>(K + tok * a.sx_l + row);
                    const f32x4 qv = ld4<T>(Q + tok * a.sx_l + row);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float at = fexp2(gv[r] * LOG2E);
#pragma unroll
                        for (int ct = 0; ct < NCT; ++ct) {
                            S[ct][i][r] = at * S[ct][i][r] + kv[r] * vv[ct];
                            part[ct] += S[ct][i][r] * qv[r];
                        }
                    }
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    float p = part[ct];
                    p = sum_rows(p);
                    if (q4 == 0) Y[tok * a.sx_l + 16 * (NCT * w + ct) + n16] = cvt<T>(p);
                }
            }
        }
    }
    if (a.n_super == 1 && a.S_out) {
        float *dst = a.S_out + d.bh * SS;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    dst[(int64_t)(16 * i + 4 * q4 + r) * D + 16 * (NCT * w + ct) + n16] = S[ct][i][r];
    }
}

// ---------------------------------------------------------------------------
// dq walker (vector gate): forward walk with S^T[v][k] (wave w owns k tiles):
//   dq[t][k] = 2^b[t][k] ( sum_v dO[t][v] S[k][v] + sum_{s<=t} P[t][s] K^[s][k] ),
//   P[t][s] = dO_t . v_s,   S^T = diag(2^b63) (S^T + V^T K^)  (per column k),
// and r[t][k] = q[t][k] dq[t][k] into dg (read by k_dk_vg).
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), 1) k_dq_vg(SegArgs a) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>(), LDE = D + 4;
    constexpr bool SP = kSplit<T>;
    using TT = Tile<T, D, NT>;
    using GT = GTile<T, D, NT>;
    constexpr int E = TT::E, RPT = TT::RPT;
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, nat_pos order
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];   // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];   // K o 2^-b, plain, swizzled (hi)
    __shared__ __attribute__((aligned(16))) T sKl[SP ? C * LDN : 8];
    constexpr int AB = 2 * C * LDT * (int)sizeof(T), SB = GT::SCR * 4;
    __shared__ __attribute__((aligned(16))) char sPraw[AB > SB ? AB : SB];  // P hi/lo, or the gate scratch
    T *sP = reinterpret_cast<T *>(sPraw), *sPl = sP + C * LDT;
    float *scratch = reinterpret_cast<float *>(sPraw);
    __shared__ __attribute__((aligned(16))) float sEt[C * LDE];  // 2^b[t][k]
    __shared__ __attribute__((aligned(16))) float sE63[D];
    __shared__ int sFast;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    const T *dO = (const T *)a.dO + xo;
    T *dQ = (T *)a.dq + xo;
    const int64_t go = d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const float *gp = a.g + go;
    float *dgp = a.dg + go;
    const int64_t SS = (int64_t)D * D;
    const int grp = tid / TT::CB, ch0 = (tid % TT::CB) * E;

    const float *src = a.n_super == 1 ? (a.S_in ? a.S_in + d.bh * SS : nullptr)
                                      : a.wsS + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 S[NCT][NK];  // S^T[v][k]: rows v = 16i + 4 q4 + r, column k = c0 + n16
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int col = 16 * (NCT * w + ct) + n16, row = 16 * i + 4 * q4;
            S[ct][i] = src ? *reinterpret_cast<const f32x4 *>(src + (int64_t)col * D + row) : f32x4{0.f, 0.f, 0.f, 0.f};
        }

    typedef T vec4T __attribute__((ext_vector_type(4)));
    TT t1, t2, t3;
    GT tg;
    vec4T qn[NCT * 4];
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        t1.load(dO + nx, a.sx_l, tid);
        t2.load(V + nx, a.sx_l, tid);
        t3.load(K + nx, a.sx_l, tid);
        tg.load(gp + (int64_t)c * C * a.sg_l, a.sg_l, tid);
    };
    issue(0);

    for (int c = 0; c < d.nch; ++c) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
                qn[4 * ct + tt] = *reinterpret_cast<const vec4T *>(
                    Q + (int64_t)(c * C + 16 * tt + n16) * a.sx_l + 16 * (NCT * w + ct) + 4 * q4);
        __syncthreads();
        if (tid == 0) sFast = 1;
        float b[RPT][E], tot[E];
        gate_cumsum<T, D, NT>(tg, b, tot, scratch, tid);
        bool ok = true;
#pragma unroll
        for (int cc = 0; cc < E; ++cc) ok = ok && tot[cc] >= kMinChunkLog2;
        if (!ok) sFast = 0;
        {
            float f[RPT][E];
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = ok ? fexp2(-b[j][cc]) : 0.f;
            store_scaled<T, D, NT, false>(t3, f, sK, sKl, LDN, tid, SWX);
            const int r0 = t1.row0(tid);
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int u = 0; u < E / 4; ++u)
                    *reinterpret_cast<f32x4 *>(&sEt[(r0 + j) * LDE + ch0 + 4 * u]) =
                        f32x4{fexp2(b[j][4 * u]), fexp2(b[j][4 * u + 1]), fexp2(b[j][4 * u + 2]), fexp2(b[j][4 * u + 3])};
        }
        t1.store_nat(sO, LDN, tid);
        t2.store_swz(sV, LDN, tid, SWX);
        if (grp == 0) {
#pragma unroll
            for (int cc = 0; cc < E; ++cc) sE63[ch0 + cc] = fexp2(tot[cc]);
        }
        if (c + 1 < d.nch) issue(c + 1);
        __syncthreads();
        const bool fast = sFast != 0;
        __syncthreads();

        if (fast) {
            // P^T[s][t] = sum_v V[s][v] dO[t][v] on the causal tiles -> P[t][s]
            for (int i = w; i < 10; i += NW) {
                int tt, st;
                tri_tile(i, tt, st);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks)
                    mma(p, ldfrag_swz<T, LDN, SWX>(sV, swo, 16 * st, 32 * ks), ldfrag_unperm<T>(sO, LDN, 16 * tt, 32 * ks, lane));
                const int t = 16 * tt + n16;
                float v4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v4[r] = 16 * st + 4 * q4 + r <= t ? p[r] : 0.f;
                const int o = t * LDT + 16 * st + 4 * q4;
                st4_split<T>(&sP[o], &sPl[SP ? o : 0], v4);
            }
            for (int e = tid; e < 512; e += NT) {
                const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
                const int idx = tile ? (32 + rr) * LDT + 48 + cc : rr * LDT + 16 + cc;
                sP[idx] = cvt<T>(0.f);
                if constexpr (SP) sPl[idx] = cvt<T>(0.f);
            }
            __syncthreads();

            frag_t<T> kh[NCT][C / 32], kl[NCT][C / 32];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int c0 = 16 * (NCT * w + ct);
                f32x4 O[4];
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) O[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    frag_t<T> fh, fl;
                    split_acc<T>(S[ct][2 * ks], S[ct][2 * ks + 1], fh, fl);
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) mma2<T>(O[tt], fh, fl, ldfrag(sO, LDN, 16 * tt, 32 * ks, lane));
                }
#pragma unroll
                for (int ks = 0; ks < C / 32; ++ks) {
                    kh[ct][ks] = ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, c0);
                    if constexpr (SP) kl[ct][ks] = ldfragTR<T, LDN, SWX>(sKl, tro, 32 * ks, c0);
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) {
                        if (32 * ks > 16 * tt + 15) continue;
                        frag_t<T> ph = ldfrag(sP, LDT, 16 * tt, 32 * ks, lane), pl = {};
                        if constexpr (SP) pl = ldfrag(sPl, LDT, 16 * tt, 32 * ks, lane);
                        mma3<T>(O[tt], kh[ct][ks], kl[ct][ks], ph, pl);
                    }
                }
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) {
                    const int t = 16 * tt + n16;
                    const f32x4 ev = *reinterpret_cast<const f32x4 *>(&sEt[t * LDE + c0 + 4 * q4]);
                    const f32x4 dq = O[tt] * ev;
                    const int64_t tok = (int64_t)c * C + t;
                    st4(dQ + tok * a.sx_l + c0 + 4 * q4, dq[0], dq[1], dq[2], dq[3]);
                    const vec4T qv = qn[4 * ct + tt];
                    *reinterpret_cast<f32x4 *>(dgp + tok * a.sg_l + c0 + 4 * q4) =
                        f32x4{dq[0] * tof<T>(qv[0]), dq[1] * tof<T>(qv[1]), dq[2] * tof<T>(qv[2]), dq[3] * tof<T>(qv[3])};
                }
            }
            // S^T = diag_cols(2^b63) (S^T + V^T K^)
#pragma unroll
            for (int ks = 0; ks < C / 32; ++ks)
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const frag_t<T> vfr = ldfragTR<T, LDN, SWX>(sV, tro, 32 * ks, 16 * i);
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) mma2b<T>(S[ct][i], vfr, kh[ct][ks], kl[ct][ks]);
                }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const float ev = sE63[16 * (NCT * w + ct) + n16];
#pragma unroll
                for (int i = 0; i < NK; ++i) S[ct][i] *= ev;
            }
        } else {
            // token by token: S^T[v][k] = a_t[k] S^T + v_t[v] k_t[k], dq_t[k] = sum_v S^T[v][k] dO_t[v]
            for (int t = 0; t < C; ++t) {
                const int64_t tok = (int64_t)c * C + t;
                float kk[NCT], ak[NCT], qq[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int col = 16 * (NCT * w + ct) + n16;
                    kk[ct] = tof<T>(K[tok * a.sx_l + col]);
                    qq[ct] = tof<T>(Q[tok * a.sx_l + col]);
                    ak[ct] = fexp2(gp[tok * a.sg_l + col] * LOG2E);
                }
                float part[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) part[ct] = 0.f;
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const int row = 16 * i + 4 * q4;
                    const f32x4 vv = ld4<T>(V + tok * a.sx_l + row);
                    const f32x4 ov = ld4<T>(dO + tok * a.sx_l + row);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
#pragma unroll
                        for (int ct = 0; ct < NCT; ++ct) {
                            S[ct][i][r] = ak[ct] * S[ct][i][r] + vv[r] * kk[ct];
                            part[ct] += S[ct][i][r] * ov[r];
                        }
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    float p = part[ct];
                    p = sum_rows(p);
                    if (q4 == 0) {
                        const int col = 16 * (NCT * w + ct) + n16;
                        dQ[tok * a.sx_l + col] = cvt<T>(p);
                        dgp[tok * a.sg_l + col] = p * qq[ct];
                    }
                }
            }
        }
    }
    if (a.n_super == 1) {
        // <dS_out, S_out> per key channel k for dg (the state here is S_out^T)
        float *dot = a.wsDot + (int64_t)d.bh * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            const int col = 16 * (NCT * w + ct) + n16;
            float p = 0.f;
            if (a.dS_out) {
                const float *ds = a.dS_out + d.bh * SS + (int64_t)col * D;
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const f32x4 x = *reinterpret_cast<const f32x4 *>(ds + 16 * i + 4 * q4);
                    p += x[0] * S[ct][i][0] + x[1] * S[ct][i][1] + x[2] * S[ct][i][2] + x[3] * S[ct][i][3];
                }
            }
            p = sum_rows(p);
            if (q4 == 0) dot[col] = p;
        }
    }
}

// ---------------------------------------------------------------------------
// dv walker (vector gate): reverse walk with G[k][v] (wave w owns v tiles):
//   dv^T[v][s] = sum_k G[k][v] 2^b63[k] K^[s][k] + sum_t dO^T[v][t] A^T[s][t]
//   G = diag(2^b63) G + Q~^T dO
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), 1) k_dv_vg(SegArgs a) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplit<T>;
    using TT = Tile<T, D, NT>;
    using GT = GTile<T, D, NT>;
    constexpr int E = TT::E, RPT = TT::RPT;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // Q o 2^b, plain, swizzled (hi)
    __shared__ __attribute__((aligned(16))) T sQl[SP ? C * LDN : 8];
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];   // K o 2^-b, nat_pos order (hi)
    __shared__ __attribute__((aligned(16))) T sKl[SP ? C * LDN : 8];
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, plain, swizzled
    constexpr int AB = 2 * C * LDT * (int)sizeof(T), SB = GT::SCR * 4;
    __shared__ __attribute__((aligned(16))) char sAraw[AB > SB ? AB : SB];  // A^T hi/lo, or the gate scratch
    T *sAT = reinterpret_cast<T *>(sAraw), *sATl = sAT + C * LDT;
    float *scratch = reinterpret_cast<float *>(sAraw);
    __shared__ __attribute__((aligned(16))) float sE63[D];
    __shared__ int sFast;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *dO = (const T *)a.dO + xo;
    T *dV = (T *)a.dv + xo;
    const float *gp = a.g + d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const int64_t SS = (int64_t)D * D;
    const int grp = tid / TT::CB, ch0 = (tid % TT::CB) * E;

    const float *gsrc = a.n_super == 1 ? (a.dS_out ? a.dS_out + d.bh * SS : nullptr)
                                       : a.wsE + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 G[NCT][NK];  // G[k][v]: rows k = 16i + 4 q4 + r, column v = c0 + n16
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                G[ct][i][r] = gsrc ? gsrc[(int64_t)(16 * i + 4 * q4 + r) * D + 16 * (NCT * w + ct) + n16] : 0.f;

    TT t1, t2, t3;
    GT tg;
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        t1.load(Q + nx, a.sx_l, tid);
        t2.load(K + nx, a.sx_l, tid);
        t3.load(dO + nx, a.sx_l, tid);
        tg.load(gp + (int64_t)c * C * a.sg_l, a.sg_l, tid);
    };
    issue(d.nch - 1);

    for (int c = d.nch - 1; c >= 0; --c) {
        __syncthreads();
        if (tid == 0) sFast = 1;
        float b[RPT][E], tot[E];
        gate_cumsum<T, D, NT>(tg, b, tot, scratch, tid);
        bool ok = true;
#pragma unroll
        for (int cc = 0; cc < E; ++cc) ok = ok && tot[cc] >= kMinChunkLog2;
        if (!ok) sFast = 0;
        {
            float f[RPT][E];
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = fexp2(b[j][cc]);
            store_scaled<T, D, NT, false>(t1, f, sQ, sQl, LDN, tid, SWX);
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = ok ? fexp2(-b[j][cc]) : 0.f;
            store_scaled<T, D, NT, true>(t2, f, sK, sKl, LDN, tid, SWX);
        }
        t3.store_swz(sO, LDN, tid, SWX);
        if (grp == 0) {
#pragma unroll
            for (int cc = 0; cc < E; ++cc) sE63[ch0 + cc] = fexp2(tot[cc]);
        }
        if (c > 0) issue(c - 1);
        __syncthreads();
        const bool fast = sFast != 0;
        __syncthreads();

        if (fast) {
            // A^T[s][t]: P[t][s] = sum_ch Q~[t][ch] K^[s][ch] on the causal tiles
            for (int i = w; i < 10; i += NW) {
                int tt, st;
                tri_tile(i, tt, st);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    const frag_t<T> qh = ldfrag_swz<T, LDN, SWX>(sQ, swo, 16 * tt, 32 * ks);
                    const frag_t<T> kh = ldfrag_unperm<T>(sK, LDN, 16 * st, 32 * ks, lane);
                    frag_t<T> ql = {}, kl = {};
                    if constexpr (SP) {
                        ql = ldfrag_swz<T, LDN, SWX>(sQl, swo, 16 * tt, 32 * ks);
                        kl = ldfrag_unperm<T>(sKl, LDN, 16 * st, 32 * ks, lane);
                    }
                    mma3<T>(p, qh, ql, kh, kl);
                }
                const int s = 16 * st + n16;
                float v4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v4[r] = s <= 16 * tt + 4 * q4 + r ? p[r] : 0.f;
                const int o = s * LDT + 16 * tt + 4 * q4;
                st4_split<T>(&sAT[o], &sATl[SP ? o : 0], v4);
            }
            for (int e = tid; e < 512; e += NT) {
                const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
                const int idx = tile ? (48 + rr) * LDT + 32 + cc : (16 + rr) * LDT + cc;
                sAT[idx] = cvt<T>(0.f);
                if constexpr (SP) sATl[idx] = cvt<T>(0.f);
            }
            __syncthreads();

            frag_t<T> of[NCT][C / 32];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int c0 = 16 * (NCT * w + ct);
                f32x4 DV[4];
#pragma unroll
                for (int st = 0; st < 4; ++st) DV[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    // G fragment scaled by 2^b63 at its contraction rows k (nat_pos order)
                    const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&sE63[32 * ks + 4 * q4]);
                    const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&sE63[32 * ks + 16 + 4 * q4]);
                    float x[8];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        x[r] = G[ct][2 * ks][r] * e0[r];
                        x[4 + r] = G[ct][2 * ks + 1][r] * e1[r];
                    }
                    frag_t<T> gh, gl;
                    split8<T>(x, gh, gl);
#pragma unroll
                    for (int st = 0; st < 4; ++st) {
                        frag_t<T> khf = ldfrag(sK, LDN, 16 * st, 32 * ks, lane), klf = {};
                        if constexpr (SP) klf = ldfrag(sKl, LDN, 16 * st, 32 * ks, lane);
                        mma3<T>(DV[st], gh, gl, khf, klf);
                    }
                }
#pragma unroll
                for (int ks = 0; ks < C / 32; ++ks) of[ct][ks] = ldfragTR<T, LDN, SWX>(sO, tro, 32 * ks, c0);
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int ks = st / 2; ks < C / 32; ++ks) {
                        mma(DV[st], of[ct][ks], ldfrag(sAT, LDT, 16 * st, 32 * ks, lane));
                        if constexpr (SP) mma(DV[st], of[ct][ks], ldfrag(sATl, LDT, 16 * st, 32 * ks, lane));
                    }
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    st4(dV + ((int64_t)c * C + 16 * st + n16) * a.sx_l + c0 + 4 * q4, DV[st][0], DV[st][1], DV[st][2],
                        DV[st][3]);
            }
            // G = diag(2^b63) G + Q~^T dO
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const f32x4 ev = *reinterpret_cast<const f32x4 *>(&sE63[16 * i + 4 * q4]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) G[ct][i] *= ev;
            }
#pragma unroll
            for (int ks = 0; ks < C / 32; ++ks)
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const frag_t<T> qh = ldfragTR<T, LDN, SWX>(sQ, tro, 32 * ks, 16 * i);
                    frag_t<T> ql = {};
                    if constexpr (SP) ql = ldfragTR<T, LDN, SWX>(sQl, tro, 32 * ks, 16 * i);
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) mma2<T>(G[ct][i], qh, ql, of[ct][ks]);
                }
        } else {
            // token by token, t descending: G += q_t dO_t^T; dv_t = G^T k_t; G = diag(a_t) G
            for (int t = C - 1; t >= 0; --t) {
                const int64_t tok = (int64_t)c * C + t;
                float ov[NCT], part[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    ov[ct] = tof<T>(dO[tok * a.sx_l + 16 * (NCT * w + ct) + n16]);
                    part[ct] = 0.f;
                }
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const int row = 16 * i + 4 * q4;
                    const f32x4 qv = ld4<T>(Q + tok * a.sx_l + row);
                    const f32x4 kv = ld4<T>(K + tok * a.sx_l + row);
                    const f32x4 gv = *reinterpret_cast<const f32x4 *>(gp + tok * a.sg_l + row);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float at = fexp2(gv[r] * LOG2E);
#pragma unroll
                        for (int ct = 0; ct < NCT; ++ct) {
                            const float gg = G[ct][i][r] + qv[r] * ov[ct];
                            part[ct] += gg * kv[r];
                            G[ct][i][r] = at * gg;
                        }
                    }
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    float p = part[ct];
                    p = sum_rows(p);
                    if (q4 == 0) dV[tok * a.sx_l + 16 * (NCT * w + ct) + n16] = cvt<T>(p);
                }
            }
        }
    }
    if (a.n_super == 1 && a.dS_in) {
        float *dst = a.dS_in + d.bh * SS;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    dst[(int64_t)(16 * i + 4 * q4 + r) * D + 16 * (NCT * w + ct) + n16] = G[ct][i][r];
    }
}

// ---------------------------------------------------------------------------
// dk walker (vector gate): reverse walk with G^T[v][k] (wave w owns k tiles):
//   dk[s][k] = 2^-b[s][k] ( 2^b63[k] sum_v G^T[v][k] V[s][v] + sum_t Q~[t][k] P^T[s][t] ),
//   P[t][s] = dO_t . v_s,  G^T = diag_cols(2^b63) G^T + dO^T Q~,
//   dg[t][k] = sum_{t' >= t in superchunk} (q dq - k dk)[t'][k] + <G_{J+1}, S_{J+1}>[k].
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), 1) k_dk_vg(SegArgs a) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>(), LDE = D + 4;
    constexpr bool SP = kSplit<T>;
    using TT = Tile<T, D, NT>;
    using GT = GTile<T, D, NT>;
    constexpr int E = TT::E, RPT = TT::RPT;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // Q o 2^b, plain, swizzled (hi)
    __shared__ __attribute__((aligned(16))) T sQl[SP ? C * LDN : 8];
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];   // nat_pos order
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, plain, swizzled
    __shared__ __attribute__((aligned(16))) T sKr[C * LDN];  // k, plain
    constexpr int AB = 2 * C * LDT * (int)sizeof(T), SB = GT::SCR * 4;
    __shared__ __attribute__((aligned(16))) char sPraw[AB > SB ? AB : SB];  // P^T hi/lo, or the gate scratch
    T *sPT = reinterpret_cast<T *>(sPraw), *sPTl = sPT + C * LDT;
    float *scratch = reinterpret_cast<float *>(sPraw);
    __shared__ __attribute__((aligned(16))) float sEi[C * LDE];  // 2^-b[s][k]
    __shared__ __attribute__((aligned(16))) float sE63[D];
    __shared__ int sFast;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    const T *dO = (const T *)a.dO + xo;
    T *dK = (T *)a.dk + xo;
    const int64_t go = d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const float *gp = a.g + go;
    float *dgp = a.dg + go;
    const int64_t SS = (int64_t)D * D;
    const int grp = tid / TT::CB, ch0 = (tid % TT::CB) * E;

    const float *gsrc = a.n_super == 1 ? (a.dS_out ? a.dS_out + d.bh * SS : nullptr)
                                       : a.wsE + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 GTr[NCT][NK];  // G^T[v][k]: rows v = 16i + 4 q4 + r, column k = c0 + n16
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int col = 16 * (NCT * w + ct) + n16;
            GTr[ct][i] = gsrc ? *reinterpret_cast<const f32x4 *>(gsrc + (int64_t)col * D + 16 * i + 4 * q4)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    // decay gradient carried in from later tokens, for this lane's channels k = c0 + 4 q4 + r
    f32x4 carry[NCT];
    {
        const float *dot = a.wsDot + ((int64_t)d.bh * a.n_super + d.J) * D;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) carry[ct] = *reinterpret_cast<const f32x4 *>(dot + 16 * (NCT * w + ct) + 4 * q4);
    }

    TT t1, t2, t3, t4;
    GT tg;
    f32x4 rn[NCT][4];  // q o dq (from the dq walk) at this lane's (s, k)
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        t1.load(Q + nx, a.sx_l, tid);
        t2.load(V + nx, a.sx_l, tid);
        t3.load(dO + nx, a.sx_l, tid);
        t4.load(K + nx, a.sx_l, tid);
        tg.load(gp + (int64_t)c * C * a.sg_l, a.sg_l, tid);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st)
                rn[ct][st] = *reinterpret_cast<const f32x4 *>(dgp + ((int64_t)c * C + 16 * st + n16) * a.sg_l +
                                                             16 * (NCT * w + ct) + 4 * q4);
    };
    issue(d.nch - 1);

    for (int c = d.nch - 1; c >= 0; --c) {
        f32x4 rc[NCT][4];
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st) rc[ct][st] = rn[ct][st];
        __syncthreads();
        if (tid == 0) sFast = 1;
        float b[RPT][E], tot[E];
        gate_cumsum<T, D, NT>(tg, b, tot, scratch, tid);
        bool ok = true;
#pragma unroll
        for (int cc = 0; cc < E; ++cc) ok = ok && tot[cc] >= kMinChunkLog2;
        if (!ok) sFast = 0;
        {
            float f[RPT][E];
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int cc = 0; cc < E; ++cc) f[j][cc] = fexp2(b[j][cc]);
            store_scaled<T, D, NT, false>(t1, f, sQ, sQl, LDN, tid, SWX);
            const int r0 = t1.row0(tid);
#pragma unroll
            for (int j = 0; j < RPT; ++j)
#pragma unroll
                for (int u = 0; u < E / 4; ++u)
                    *reinterpret_cast<f32x4 *>(&sEi[(r0 + j) * LDE + ch0 + 4 * u]) =
                        ok ? f32x4{fexp2(-b[j][4 * u]), fexp2(-b[j][4 * u + 1]), fexp2(-b[j][4 * u + 2]),
                                   fexp2(-b[j][4 * u + 3])}
                           : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        t2.store_nat(sV, LDN, tid);
        t3.store_swz(sO, LDN, tid, SWX);
        {
            typedef T vecE __attribute__((ext_vector_type(E)));
            const int r0 = t4.row0(tid);
#pragma unroll
            for (int j = 0; j < RPT; ++j) *reinterpret_cast<vecE *>(&sKr[(r0 + j) * LDN + ch0]) = t4.r[j];
        }
        if (grp == 0) {
#pragma unroll
            for (int cc = 0; cc < E; ++cc) sE63[ch0 + cc] = fexp2(tot[cc]);
        }
        if (c > 0) issue(c - 1);
        __syncthreads();
        const bool fast = sFast != 0;
        __syncthreads();

        if (fast) {
            // P^T[s][t]: P[t][s] = sum_v dO[t][v] V[s][v] on the causal tiles
            for (int i = w; i < 10; i += NW) {
                int tt, st;
                tri_tile(i, tt, st);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks)
                    mma(p, ldfrag_swz<T, LDN, SWX>(sO, swo, 16 * tt, 32 * ks), ldfrag_unperm<T>(sV, LDN, 16 * st, 32 * ks, lane));
                const int s = 16 * st + n16;
                float v4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v4[r] = s <= 16 * tt + 4 * q4 + r ? p[r] : 0.f;
                const int o = s * LDT + 16 * tt + 4 * q4;
                st4_split<T>(&sPT[o], &sPTl[SP ? o : 0], v4);
            }
            for (int e = tid; e < 512; e += NT) {
                const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
                const int idx = tile ? (48 + rr) * LDT + 32 + cc : (16 + rr) * LDT + cc;
                sPT[idx] = cvt<T>(0.f);
                if constexpr (SP) sPTl[idx] = cvt<T>(0.f);
            }
            __syncthreads();

            frag_t<T> qh[NCT][C / 32], ql[NCT][C / 32];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const int c0 = 16 * (NCT * w + ct);
                f32x4 X1[4], X2[4];
#pragma unroll
                for (int st = 0; st < 4; ++st) X1[st] = X2[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    frag_t<T> fh, fl;
                    split_acc<T>(GTr[ct][2 * ks], GTr[ct][2 * ks + 1], fh, fl);
#pragma unroll
                    for (int st = 0; st < 4; ++st) mma2<T>(X1[st], fh, fl, ldfrag(sV, LDN, 16 * st, 32 * ks, lane));
                }
#pragma unroll
                for (int ks = 0; ks < C / 32; ++ks) {
                    qh[ct][ks] = ldfragTR<T, LDN, SWX>(sQ, tro, 32 * ks, c0);
                    if constexpr (SP) ql[ct][ks] = ldfragTR<T, LDN, SWX>(sQl, tro, 32 * ks, c0);
                }
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int ks = st / 2; ks < C / 32; ++ks) {
                        frag_t<T> ph = ldfrag(sPT, LDT, 16 * st, 32 * ks, lane), pl = {};
                        if constexpr (SP) pl = ldfrag(sPTl, LDT, 16 * st, 32 * ks, lane);
                        mma3<T>(X2[st], qh[ct][ks], ql[ct][ks], ph, pl);
                    }
                // dk = 2^-b (2^b63 X1 + X2); k o dk; dg suffix over the chunk
                const f32x4 e63 = *reinterpret_cast<const f32x4 *>(&sE63[c0 + 4 * q4]);
                f32x4 y[4];
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const int s = 16 * st + n16;
                    const f32x4 ei = *reinterpret_cast<const f32x4 *>(&sEi[s * LDE + c0 + 4 * q4]);
                    const f32x4 dk = (X1[st] * e63 + X2[st]) * ei;
                    st4(dK + ((int64_t)c * C + s) * a.sx_l + c0 + 4 * q4, dk[0], dk[1], dk[2], dk[3]);
                    const f32x4 kv = ld4f(&sKr[s * LDN + c0 + 4 * q4]);
                    y[st] = rc[ct][st] - kv * dk;
                }
                // suffix sums over s = 16 st + n16 for each of the lane's 4 channels
                f32x4 tot4[4];
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float x = y[st][r];
                        x += dpp_row_shl<1>(x);
                        x += dpp_row_shl<2>(x);
                        x += dpp_row_shl<4>(x);
                        x += dpp_row_shl<8>(x);
                        y[st][r] = x;
                        tot4[st][r] = __shfl(x, lane & 48, 64);
                    }
                f32x4 later = carry[ct];
#pragma unroll
                for (int st = 3; st >= 0; --st) {
                    const f32x4 dg = y[st] + later;
                    *reinterpret_cast<f32x4 *>(dgp + ((int64_t)c * C + 16 * st + n16) * a.sg_l + c0 + 4 * q4) = dg;
                    later += tot4[st];
                }
                carry[ct] = later;
            }
            // G^T = diag_cols(2^b63) G^T + dO^T Q~
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const float ev = sE63[16 * (NCT * w + ct) + n16];
#pragma unroll
                for (int i = 0; i < NK; ++i) GTr[ct][i] *= ev;
            }
#pragma unroll
            for (int ks = 0; ks < C / 32; ++ks)
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const frag_t<T> of = ldfragTR<T, LDN, SWX>(sO, tro, 32 * ks, 16 * i);
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) mma2b<T>(GTr[ct][i], of, qh[ct][ks], ql[ct][ks]);
                }
        } else {
            // token by token, t descending: G^T += dO_t q_t^T; dk_t = G^T^T v_t; G^T = G^T diag(a_t).
            // The running dg of column k = c0 + n16 lives in acc[ct] of every lane of that column.
            float acc[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = __shfl(carry[ct][r], (n16 >> 2) << 4, 64);
                const int rr = n16 & 3;
                acc[ct] = rr == 0 ? v[0] : rr == 1 ? v[1] : rr == 2 ? v[2] : v[3];
            }
            for (int t = C - 1; t >= 0; --t) {
                const int64_t tok = (int64_t)c * C + t;
                float qq[NCT], kk[NCT], ak[NCT], part[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int col = 16 * (NCT * w + ct) + n16;
                    qq[ct] = tof<T>(Q[tok * a.sx_l + col]);
                    kk[ct] = tof<T>(K[tok * a.sx_l + col]);
                    ak[ct] = fexp2(gp[tok * a.sg_l + col] * LOG2E);
                    part[ct] = 0.f;
                }
#pragma unroll
                for (int i = 0; i < NK; ++i) {
                    const int row = 16 * i + 4 * q4;
                    const f32x4 ov = ld4<T>(dO + tok * a.sx_l + row);
                    const f32x4 vv = ld4<T>(V + tok * a.sx_l + row);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
#pragma unroll
                        for (int ct = 0; ct < NCT; ++ct) {
                            const float gg = GTr[ct][i][r] + ov[r] * qq[ct];
                            part[ct] += gg * vv[r];
                            GTr[ct][i][r] = ak[ct] * gg;
                        }
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    float p = part[ct];
                    p = sum_rows(p);  // dk_t[col], every lane of the column
                    const int col = 16 * (NCT * w + ct) + n16;
                    acc[ct] += dgp[tok * a.sg_l + col] - kk[ct] * p;  // + r_t - k_t dk_t
                    if (q4 == 0) {
                        dK[tok * a.sx_l + col] = cvt<T>(p);
                        dgp[tok * a.sg_l + col] = acc[ct];
                    }
                }
            }
            // bring the per-column running sums back to the carry layout (k = c0 + 4 q4 + r)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int r = 0; r < 4; ++r) carry[ct][r] = __shfl(acc[ct], 4 * q4 + r, 64);
        }
    }
}

// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t launch_vg_td(int kind, const SegArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int NCT = 2, NT = 64 * D / (16 * NCT);
    constexpr int NC1 = 1, NT1 = 64 * D / 16;  // fwd and dk/dv walks: one 16-column tile per wave
    const dim3 grid((unsigned)((int64_t)a.B * a.H * a.n_super));
    switch (kind) {
    case SF_K_FWD_PREP: hipExtLaunchKernelGGL((k_prep_vg<T, D, NCT, false>), grid, dim3(NT), 0, s, e0, e1, 0, a); break;
    case SF_K_FWD_OUT: hipExtLaunchKernelGGL((k_walk_vg<T, D, NC1>), grid, dim3(NT1), 0, s, e0, e1, 0, a); break;
    case SF_K_BWD_PREP:  // the replay of D_J is skipped when the forward kept the states
        if (a.ckpt) {
            hipExtLaunchKernelGGL((k_prep_vg<T, D, NCT, true>), grid, dim3(NT), 0, s, e0, e1, 0, a);
        } else {
            hipExtLaunchKernelGGL((k_prep_vg_bwd<T, D, NCT>), dim3(2 * grid.x), dim3(NT), 0, s, e0, e1, 0, a);
        }
        break;
    case SF_K_BWD_DQ: hipExtLaunchKernelGGL((k_dq_vg<T, D, NCT>), grid, dim3(NT), 0, s, e0, e1, 0, a); break;
    case SF_K_BWD_DKV:
        hipExtLaunchKernelGGL((k_dv_vg<T, D, NC1>), grid, dim3(NT1), 0, s, e0, nullptr, 0, a);
        hipExtLaunchKernelGGL((k_dk_vg<T, D, NC1>), grid, dim3(NT1), 0, s, nullptr, e1, 0, a);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_kernel_vg(int kind, int io, int D, const SegArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (io == SF_BF16 && D == 128) return launch_vg_td<__bf16, 128>(kind, a, s, e0, e1);
    if (io == SF_BF16 && D == 64) return launch_vg_td<__bf16, 64>(kind, a, s, e0, e1);
    if (io == SF_F32 && D == 64) return launch_vg_td<float, 64>(kind, a, s, e0, e1);
    return hipErrorInvalidValue;
}

}  // namespace sf
