// sf_kernels.hip -- gfx950 kernels of the segmented gated linear recurrence.
//
// Per (batch, head) the recurrence S_t = a_t S_{t-1} + k_t v_t^T, o_t = S_t^T q_t
// (paper Sec. 2.1, Eq. 1) is evaluated in the chunkwise form of Sec. 2.2 (Eq. 2):
// a segment of L tokens is cut into kernel-level chunks of C = 64 tokens and
// into "superchunks" of ts tokens (a multiple of C) at which the state is
// materialised.  With b_j the chunk-local inclusive cumulative log-decay,
//   intra:  A = (Q K^T) o M,  M[t][s] = exp(b_t - b_s) [s <= t]
//   out:    O = diag(exp(b)) Q S_c + A V
//   state:  S_{c+1} = exp(b_63) S_c + (K o exp(b_63 - b))^T V
// Every exponent is <= 0 (g <= 0), so no factor can overflow.
//
// Kernels (one workgroup of D/16 waves per (batch, head, superchunk); wave w
// owns the 16 state columns [16w, 16w+16)):
//   k_prep<.., EONLY=false> Pre: superchunk state contribution D_J and its decay
//                           (in the backward too, as the replay of the forward's)
//   k_scan<false>           ST:  S_{J+1} = Gamma_J S_J + D_J (fp32), S_out
//   k_walk<.., DQ=false>    Out: walk the chunks from S_J, write o
//   k_prep<.., EONLY=true>  the state-gradient contribution E_J
//   k_prep_bwd              the backward's replay of D_J and its E_J in one launch
//   k_scan<true>            ST + STB: S_J forward, G_{J+1} backward, dS_in,
//                           <G_{J+1}, S_{J+1}> partials for dg
//   k_walk<.., DQ=true>     dq by a forward walk; also q.dq per token
//   k_bwd_dkv               dk, dv, dg by a reverse walk of the state gradient
// A segment that fits in one superchunk skips prep and scan: the walkers start
// from S_in / dS_out directly and produce S_out / dS_in themselves.
#include "sf_chunk.hpp"

namespace sf {

constexpr int SCAN_NT = 256;

// state column tiles per wave of the prep kernels (forward, backward) and of
// the chunk walkers: 2 gives D/32 waves per workgroup, twice the reuse of every
// shared operand fragment and workgroups small enough for two per CU
#ifndef SF_NCT_PREP
#define SF_NCT_PREP 2
#endif
#ifndef SF_NCT_WALK
#define SF_NCT_WALK 2
#endif
#ifndef SF_NCT_DKV
#define SF_NCT_DKV 2
#endif

// ---------------------------------------------------------------------------
// Pre: per superchunk, D_J = sum_c (decay after c) (K~_c)^T V_c (forward, and
// its replay in the backward), or E_J = sum_t exp(B_t) q_t dO_t^T (backward,
// B superchunk-local, inclusive).  Wave w owns NCT state column tiles.  The key
// (query) tile is read through transposing loads as the exact shared operand;
// the per-token factor goes on the wave's own value (dO) columns, split hi/lo:
//   D[k][col] = gam D[k][col] + sum_s K[s][k] (exp2(b63 - b_s) V[s][col])
//   E[k][col] =                 sum_t Q[t][k] (exp2(off + b_t) dO[t][col])
// with off the log2 decay of the superchunk's earlier chunks (E: EONLY).
// One superchunk (item) of either summary; the LDS tiles come from the kernel:
// sK (q for E) and sV (dO for E), C x (D + pad), and se, the per-token factor.
template <typename T, int D, int NCT, bool EONLY>
__device__ __forceinline__ void prep_item(const SegArgs &a, int item, T *sK, T *sV, float *se) {
    constexpr int NW = D / (16 * NCT), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), SWX = swx<T, D>();
    constexpr bool SPD = kSplitDecay<T>;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const Decode d = decode(a, item);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *K = (const T *)(EONLY ? a.q : a.k) + xo;
    const T *V = (const T *)(EONLY ? a.dO : a.v) + xo;
    const float *gp = a.g + d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;

    f32x4 Ds[NCT][NK];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) Ds[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};

    Tile<T, D, NT> tk, tv;
    float gl;
    auto issue = [&](int c) {
        const int64_t nx = (int64_t)c * C * a.sx_l;
        tk.load(K + nx, a.sx_l, tid);
        tv.load(V + nx, a.sx_l, tid);
        gl = gp[(c * C + lane) * a.sg_l];
    };
    issue(0);
    float off = 0.f;  // log2 decay of the superchunk's earlier chunks

    const unsigned par = pair_parity(a.n_cu);
    for (int c = 0; c < d.nch; ++c) {
        pair_turn(par);
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        __syncthreads();
        if (w == 0) se[lane] = EONLY ? fexp2(off + b2) : fexp2(b63 - b2);
        tk.store_swz(sK, LDN, tid, SWX);
        tv.store_swz(sV, LDN, tid, SWX);
        if (c + 1 < d.nch) issue(c + 1);
        __syncthreads();
        if constexpr (!EONLY) {
            const float gam = fexp2(b63);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int i = 0; i < NK; ++i) Ds[ct][i] *= gam;
        }
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const int s0 = 32 * ks + 8 * q4;
            const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&se[s0]);
            const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&se[s0 + 4]);
            const float ev[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
            frag_t<T> vh[NCT], vl[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
                split_scaled<T, SPD>(ldfragTR<T, LDN, SWX>(sV, tro, 32 * ks, 16 * (NCT * w + ct)), ev, vh[ct], vl[ct]);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> kf = ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, 16 * i);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) mma2b<T, SPD>(Ds[ct][i], kf, vh[ct], vl[ct]);
            }
        }
        off += b63;
    }
    const int64_t so = ((int64_t)d.bh * a.n_super + d.J) * D * D;
    float *dst = EONLY ? a.wsE : a.wsS;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int c0 = 16 * (NCT * w + ct);
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[so + (int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = Ds[ct][i][r];
    }
    if (!EONLY && tid == 0) a.wsLg[(int64_t)d.bh * a.n_super + d.J] = off;
}

template <typename T, int D, int NCT, bool EONLY>
__global__ void __launch_bounds__(64 * D / (16 * NCT), sizeof(T) == 2 ? 2 : 1) k_prep(SegArgs a) {
    constexpr int LDN = D + pad<T>();
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];
    __shared__ __attribute__((aligned(16))) float se[C];
    prep_item<T, D, NCT, EONLY>(a, (int)blockIdx.x, sK, sV, se);
}

// The backward's two summaries in one launch: workgroups [0, n) replay D_J,
// [n, 2n) form E_J (n = B H n_super).  Neither waits for the other, and the
// last dispatch round of one overlaps the other's work.
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(64 * D / (16 * NCT), sizeof(T) == 2 ? 2 : 1) k_prep_bwd(SegArgs a) {
    constexpr int LDN = D + pad<T>();
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];
    __shared__ __attribute__((aligned(16))) float se[C];
    const int n = (int)(gridDim.x / 2), item = (int)blockIdx.x;
    if (item < n) prep_item<T, D, NCT, false>(a, item, sK, sV, se);
    else prep_item<T, D, NCT, true>(a, item - n, sK, sV, se);
}

// ---------------------------------------------------------------------------
// ST (and STB): fp32 scan over superchunk summaries, 4 state elements per
// thread; grid = B*H*(D*D/1024).  Forward: slot J of wsS is replaced by S_J
// (state entering superchunk J).  Backward additionally walks J downwards:
// slot J of wsE is replaced by G_{J+1} (gradient of the state leaving J) and
// <G_{J+1}, S_{J+1}> goes to wsDot: scalar gate as wave partials at
// [(bh, J)][part*4 + wave], vector gate (VG) per key row at [(bh, J)][row].
// VG: the superchunk decay is per key row (wsLg[(bh, J)][row]); a thread's 4
// elements lie in one row.
// Kept states: the forward also writes the final state to wsSn; a backward
// with a.ckpt set finds S_J already in wsS and the final state in wsSn, and
// runs the backward half only.
template <bool BWD, bool VG>
__global__ void __launch_bounds__(SCAN_NT) k_scan(SegArgs a, int D) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int parts = D * D / 1024;
    const int part = blockIdx.x % parts;
    const int64_t bh = blockIdx.x / parts;
    const int64_t SS = (int64_t)D * D;
    const int64_t e = (int64_t)(part * SCAN_NT + tid) * 4;
    const int row = (int)(e / D);
    const int n = a.n_super;
    float *Sb = a.wsS + bh * n * SS + e;
    const int LS = VG ? D : 1;  // wsLg entries per superchunk
    const float *lg = a.wsLg + bh * n * LS + (VG ? row : 0);

    // The chain over J is sequential; its loads are not.  Superchunks go in
    // batches of SB, double-buffered: the loads of the next batch are in flight
    // while the current one is applied (slot indices stay compile-time).
    constexpr int SB = 8;
    f32x4 S = a.S_in ? *reinterpret_cast<const f32x4 *>(a.S_in + bh * SS + e) : f32x4{0.f, 0.f, 0.f, 0.f};
    if (BWD && a.ckpt) {
        S = *reinterpret_cast<const f32x4 *>(a.wsSn + bh * SS + e);
    } else {
        f32x4 dd[2][SB];
        float f[2][SB];
        auto fetch = [&](int slot, int J0) {
#pragma unroll
            for (int u = 0; u < SB; ++u)
                if (J0 + u < n) {
                    dd[slot][u] = *reinterpret_cast<const f32x4 *>(Sb + (int64_t)(J0 + u) * SS);
                    f[slot][u] = fexp2(lg[(J0 + u) * LS]);
                }
        };
        // slot J of wsS: D_J in, S_J out (this thread reads each element before it writes it)
        auto apply = [&](int slot, int J0) {
#pragma unroll
            for (int u = 0; u < SB; ++u)
                if (J0 + u < n) {
                    *reinterpret_cast<f32x4 *>(Sb + (int64_t)(J0 + u) * SS) = S;
                    S = f[slot][u] * S + dd[slot][u];
                }
        };
        fetch(0, 0);
        for (int J0 = 0; J0 < n; J0 += 2 * SB) {
            if (J0 + SB < n) fetch(1, J0 + SB);
            apply(0, J0);
            if (J0 + 2 * SB < n) fetch(0, J0 + 2 * SB);
            if (J0 + SB < n) apply(1, J0 + SB);
        }
    }
    if constexpr (!BWD) {
        if (a.S_out) *reinterpret_cast<f32x4 *>(a.S_out + bh * SS + e) = S;
        if (a.wsSn) *reinterpret_cast<f32x4 *>(a.wsSn + bh * SS + e) = S;
    } else {
        const int ndot = VG ? D : D * D / 256;
        float *Eb = a.wsE + bh * n * SS + e;
        f32x4 G = a.dS_out ? *reinterpret_cast<const f32x4 *>(a.dS_out + bh * SS + e)
                           : f32x4{0.f, 0.f, 0.f, 0.f};
        f32x4 Sn = S;  // S_{J+1} for J = n-1 is S_out
        f32x4 E[2][SB], Sj[2][SB];
        float f[2][SB];
        // batch starting at J0 going down: superchunks J0, J0-1, ..., J0-SB+1
        auto fetch = [&](int slot, int J0) {
#pragma unroll
            for (int u = 0; u < SB; ++u)
                if (J0 - u >= 0) {
                    E[slot][u] = *reinterpret_cast<const f32x4 *>(Eb + (int64_t)(J0 - u) * SS);
                    Sj[slot][u] = *reinterpret_cast<const f32x4 *>(Sb + (int64_t)(J0 - u) * SS);
                    f[slot][u] = fexp2(lg[(J0 - u) * LS]);
                }
        };
        auto apply = [&](int slot, int J0) {
#pragma unroll
            for (int u = 0; u < SB; ++u)
                if (J0 - u >= 0) {
                    const int J = J0 - u;
                    float p = G[0] * Sn[0] + G[1] * Sn[1] + G[2] * Sn[2] + G[3] * Sn[3];
                    if constexpr (!VG) {
                        p = lane_value(wave_scan_dpp(p), 63);
                        if (lane == 0) a.wsDot[(bh * n + J) * ndot + part * 4 + w] = p;
                    } else {
                        // the D/4 threads of one row are consecutive lanes
                        for (int o = D / 8; o >= 1; o >>= 1) p += __shfl_xor(p, o, 64);
                        if ((lane & (D / 4 - 1)) == 0) a.wsDot[(bh * n + J) * ndot + row] = p;
                    }
                    *reinterpret_cast<f32x4 *>(Eb + (int64_t)J * SS) = G;
                    G = f[slot][u] * G + E[slot][u];
                    Sn = Sj[slot][u];
                }
        };
        fetch(0, n - 1);
        for (int J0 = n - 1; J0 >= 0; J0 -= 2 * SB) {
            if (J0 - SB >= 0) fetch(1, J0 - SB);
            apply(0, J0);
            if (J0 - 2 * SB >= 0) fetch(0, J0 - 2 * SB);
            if (J0 - SB >= 0) apply(1, J0 - SB);
        }
        if (a.dS_in) *reinterpret_cast<f32x4 *>(a.dS_in + bh * SS + e) = G;
    }
}

// ---------------------------------------------------------------------------
// Forward walker over the chunks of one superchunk, state in registers.
//   DQ == false (Out):  X1 = q, X2 = k, X3 = v, state S[k][v];   writes o.
//   DQ == true  (OG):   X1 = dO, X2 = v, X3 = k, state S^T[v][k]; writes dq
//                       and r_t = q_t . dq_t into dg (read back by k_bwd_dkv).
// Wave w owns NCT state column tiles.  The state lives as MFMA accumulators:
// row tile i of lane l holds rows 16i+4*(l/16)+r of column c0+l%16, which is an
// A-operand fragment of the transposed state once two lane-row swaps put its
// channels in plain order (split_acc_plain), so X1 S needs no LDS round trip
// for S.  LDS holds the three input tiles in natural [token][channel] layout
// only: X1 plain and unswizzled (whole 16-byte fragment reads, conflict-free),
// X2 and X3 plain and swizzled for the transposing loads that feed the state
// update (X2^T, the exact shared operand) and the value side (X3^T, decayed per
// token and split hi/lo in registers by the wave that owns those columns).
// The score tiles XOR their 16-byte blocks by bit 2 of the row and the output
// staging tile uses a 16-byte-odd pitch: both halve the bank conflicts of the
// 8-byte accumulator-row writes.
// CS > 1 (output walk only): the state's columns are split over CS workgroups
// per item, each staging the whole chunk and forming the scores but keeping
// and writing only its D / CS columns; for launches that would leave half the
// CUs idle.
// The CS workgroups of an item lie 8 apart in dispatch order (one XCD, so the
// second read of a tile meets L2).
template <typename T, int D, int NCT, bool DQ, int CS = 1>
__global__ void __launch_bounds__(64 * D / (16 * NCT * CS), sizeof(T) == 2 ? 2 : 1) k_walk(SegArgs a) {
    static_assert(CS == 1 || (CS == 2 && !DQ), "column split: output walk, two parts");
    constexpr int NW = D / (16 * NCT * CS), NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplitScores<T>, SPS = kSplitState<T>, SPD = kSplitDecay<T>;
    __shared__ __attribute__((aligned(16))) T sX1[C * LDN];
    __shared__ __attribute__((aligned(16))) T sX2[C * LDN];
    __shared__ __attribute__((aligned(16))) T sX3[C * LDN];
    // A[t][s] hi/lo; between chunks the same bytes stage the previous chunk's
    // output tile [token][channel] for row-contiguous global stores
    constexpr int AB = (SP ? 2 : 1) * C * LDT * (int)sizeof(T), YB = C * (D + 16 / (int)sizeof(T)) * (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) char sAraw[AB > YB ? AB : YB];
    T *const sA = reinterpret_cast<T *>(sAraw), *const sAl = SP ? sA + C * LDT : sA;
    T *const sY = reinterpret_cast<T *>(sAraw);
    constexpr int LDY = D + 16 / (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) float sb[C];   // b_t (log2, chunk-local)
    __shared__ __attribute__((aligned(16))) float sq[C];   // exp2(b_t)
    __shared__ __attribute__((aligned(16))) float se[C];   // exp2(b63 - b_t)
    __shared__ float sred[DQ ? NW * C : 1];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, q4 = lane >> 4, n16 = lane & 15;
    const int blk = (int)blockIdx.x;
    const int half = CS > 1 ? (blk >> 3) & 1 : 0, item = CS > 1 ? (blk >> 4) * 8 + (blk & 7) : blk;
    if (CS > 1 && item >= a.B * a.H * a.n_super) return;  // the last group of 8 items is ragged
    const int wc = w + NW * half;  // the wave's place among the D / (16 NCT) column owners
    const Decode d = decode(a, item);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    // bf16: the state's rows are read into the update's A operands in the order
    // that puts channels 8q..8q+7 of each 32-channel block in lane row q of the
    // accumulator pair (2m, 2m+1), the plain order of the Q.S operand: row r of
    // tile i holds channel srow(i, r), and the pair splits with no lane swaps
    constexpr bool RP = sizeof(T) == 2;
    const LaneOff tro8 = RP ? tr_off8<T, LDN, SWX>(lane) : tro;  // (tr_off8 serves 16-bit tiles only)
    auto srow = [&](int i, int r) { return RP ? 32 * (i >> 1) + 8 * q4 + 4 * (i & 1) + r : 16 * i + 4 * q4 + r; };
    // bf16 with two column tiles per wave: the state's columns (the value
    // channels of the update's own operand, read through tro8) in the order
    // that gives lane row q4 channels 32w + 8 q4 .. +7 across the two tiles of
    // the output accumulators, so its q values and its output row segments are
    // single 16-byte accesses: column n of tile ct is channel scol(ct, n)
    constexpr bool CP = RP && NCT == 2;
    auto scol = [&](int ct, int n) { return CP ? 32 * wc + 8 * (n >> 2) + 4 * ct + (n & 3) : 16 * (NCT * wc + ct) + n; };
    const int ccol0 = CP ? 32 * wc : 16 * NCT * wc, ccstep = CP ? 4 : 16;  // ldfragTR column of tile ct
    const LaneOff troc = CP ? tro8 : tro;
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *X1 = (const T *)(DQ ? a.dO : a.q) + xo;
    const T *X2 = (const T *)(DQ ? a.v : a.k) + xo;
    const T *X3 = (const T *)(DQ ? a.k : a.v) + xo;
    const T *Qd = (const T *)(DQ ? a.q : a.v) + xo;  // DQ: q for the q.dq dot
    T *Y = (T *)(DQ ? a.dq : a.o) + xo;
    const int64_t go = d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const float *gp = a.g + go;
    float *dgp = a.dg + go;
    const int64_t SS = (int64_t)D * D;

    // initial state S_J (column tiles NCT*w + ct)
    const float *src = a.n_super == 1 ? (a.S_in ? a.S_in + d.bh * SS : nullptr)
                                      : a.wsS + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 S[NCT][NK];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int col = scol(ct, n16);
            if (!src) {
                S[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};
            } else if constexpr (!DQ) {
#pragma unroll
                for (int r = 0; r < 4; ++r) S[ct][i][r] = src[(int64_t)srow(i, r) * D + col];
            } else {
                S[ct][i] = *reinterpret_cast<const f32x4 *>(src + (int64_t)col * D + srow(i, 0));
            }
        }
    typedef T vec4T __attribute__((ext_vector_type(4)));
    Tile<T, D, NT> t1, t2, t3;
    float gl;
    vec4T qn[DQ ? NCT * 4 : 1];  // DQ: q values of this lane's dq elements
    // chunk c of a token tensor is a buffer resource over its C rows: tile rows
    // at per-lane 32-bit offsets, accumulator rows (token 16tt + n16, channels
    // c0 + 4q4..) at a per-lane offset plus the uniform offset of token tile tt
    const int64_t cstep = (int64_t)C * a.sx_l;
    const uint32_t cspan = chunk_span<T, D>(a.sx_l), gspan = (uint32_t)(((C - 1) * a.sg_l + 1) * 4);
    uint32_t toff[Tile<T, D, NT>::RPT];
    Tile<T, D, NT>::offsets(toff, a.sx_l, tid);
    const uint32_t goff = (uint32_t)(lane * a.sg_l * 4);
    const uint32_t aoff = (uint32_t)((n16 * a.sx_l + (CP ? 32 * wc + 8 * q4 : 16 * NCT * wc + 4 * q4)) * (int64_t)sizeof(T));
    const uint32_t tstep = (uint32_t)(16 * a.sx_l * (int64_t)sizeof(T));
    // the next chunk's tiles go out in three batches (X1 and g at staging, X2 at
    // the start of the scores, X3 at the start of the output products), so the
    // vector-memory queue drains behind compute instead of stalling every wave
    // at one point
    auto issue1 = [&](int c) {
        t1.load_buf(buf_rsrc(X1 + c * cstep, cspan), toff, 0);
        gl = buf_ld<float>(buf_rsrc(gp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
    };
    auto issue2 = [&](int c) { t2.load_buf(buf_rsrc(X2 + c * cstep, cspan), toff, 0); };
    auto issue3 = [&](int c) { t3.load_buf(buf_rsrc(X3 + c * cstep, cspan), toff, 0); };
    auto issue_q = [&](int c) {  // DQ: q at this lane's dq elements, read after chunk c-1's dot
        const rsrc_t rq = buf_rsrc(Qd + c * cstep, cspan);
        if constexpr (CP) {  // channels 32w + 8q4 .. +7: tile 0's four, then tile 1's
            typedef T vec8T __attribute__((ext_vector_type(8)));
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const vec8T x = buf_ld<vec8T>(rq, aoff, tt * tstep);
                qn[tt] = __builtin_shufflevector(x, x, 0, 1, 2, 3);
                qn[4 + tt] = __builtin_shufflevector(x, x, 4, 5, 6, 7);
            }
        } else {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int tt = 0; tt < 4; ++tt)
                    qn[4 * ct + tt] = buf_ld<vec4T>(rq, aoff + 16 * ct * (uint32_t)sizeof(T), tt * tstep);
        }
    };
    vec4T yo[NCT][4];  // this lane's outputs of the chunk, accumulator layout
    // a chunk's outputs go registers -> LDS tile (once every wave is done with the
    // score tiles) -> whole-row 16-byte global stores early in the next chunk
    auto put_y = [&]() {
        if constexpr (CP) {  // one 16-byte row segment per token tile
            typedef T vec8T __attribute__((ext_vector_type(8)));
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
                *reinterpret_cast<vec8T *>(&sY[(16 * tt + n16) * LDY + 32 * wc + 8 * q4]) =
                    __builtin_shufflevector(yo[0][tt], yo[1][tt], 0, 1, 2, 3, 4, 5, 6, 7);
        } else {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int tt = 0; tt < 4; ++tt)
                    *reinterpret_cast<vec4T *>(&sY[(16 * tt + n16) * LDY + 16 * (NCT * wc + ct) + 4 * q4]) = yo[ct][tt];
        }
    };
    auto store_y = [&](int cp) {
        typedef typename Tile<T, D, NT>::vecE vecE;
        constexpr int E = Tile<T, D, NT>::E, CB = Tile<T, D, NT>::CB, RPT = Tile<T, D, NT>::RPT;
        const int r0 = (tid / CB) * RPT, ch = (tid % CB) * E;
        if (CS > 1 && (ch < half * (D / CS) || ch >= (half + 1) * (D / CS))) return;  // another part's columns
        const rsrc_t ry = buf_rsrc(Y + cp * cstep, cspan);
#pragma unroll
        for (int j = 0; j < RPT; ++j) buf_st(ry, toff[j], 0, *reinterpret_cast<const vecE *>(&sY[(r0 + j) * LDY + ch]));
    };
    issue1(0);
    issue2(0);
    issue3(0);
    if constexpr (DQ) issue_q(0);

    const unsigned par = pair_parity(a.n_cu);
    for (int c = 0; c < d.nch; ++c) {
        pair_turn(par);
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        __syncthreads();
        // the decay tables and (dq walk) the previous chunk's q.dq sums come from
        // the last wave, which forms no more score tiles than wave 0 (one fewer
        // with four waves)
        if (w == NW - 1) {
            sb[lane] = b2;
            sq[lane] = fexp2(b2);
            se[lane] = fexp2(b63 - b2);
        }
        t1.store_swz(sX1, LDN, tid, 0);
        t2.store_swz(sX2, LDN, tid, SWX);
        t3.store_swz(sX3, LDN, tid, SWX);
        // previous outputs out before the next loads: the wait for those loads
        // (one counter for loads and stores) then also covers these stores
        if (c > 0) store_y(c - 1);
        if (c + 1 < d.nch) issue1(c + 1);
        __syncthreads();
        if (c + 1 < d.nch) issue2(c + 1);
        if constexpr (DQ) {  // q.dq of the previous chunk, beside the scores
            if (w == NW - 1 && c > 0) {
                float r = 0.f;
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) r += sred[ww * C + lane];
                dgp[(int64_t)((c - 1) * C + lane) * a.sg_l] = r;
            }
        }

        // scores P^T[s][t] = sum_ch X2[s][ch] X1[t][ch] on the causal tiles -> A[t][s]
        for (int i = w; i < 10; i += NW) {
            int tt, st;
            tri_tile(i, tt, st);
            f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                mma(p, ldfrag_swz<T, LDN, SWX>(sX2, swo, 16 * st, 32 * ks),
                    ldfrag(sX1, LDN, 16 * tt, 32 * ks, lane));
            const int t = 16 * tt + n16;
            const float bt = sb[t];
            const f32x4 bs = *reinterpret_cast<const f32x4 *>(&sb[16 * st + 4 * q4]);
            float v4[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int s = 16 * st + 4 * q4 + r;
                v4[r] = s <= t ? p[r] * fexp2(bt - bs[r]) : 0.f;
            }
            const int o = t * LDT + ((16 * st + 4 * q4) ^ (sizeof(T) == 2 ? 8 * ((t >> 2) & 1) : 0));
            st4_split<T, SP>(&sA[o], &sAl[SP ? o : 0], v4);
        }
        // A tiles read by the A.V product but above the diagonal are zero (written
        // every chunk: the same bytes staged the previous outputs)
        for (int e = tid; e < 512; e += NT) {
            const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
            const int idx = (tile ? (32 + rr) * LDT : rr * LDT) + ((tile ? 48 + cc : 16 + cc) ^ (sizeof(T) == 2 ? 8 * ((rr >> 2) & 1) : 0));
            sA[idx] = cvt<T>(0.f);
            if constexpr (SP) sAl[idx] = cvt<T>(0.f);
        }
        __syncthreads();
        if (c + 1 < d.nch) issue3(c + 1);

        // Y^T[col][t] = exp2(b_t) sum_m S[m][col] X1[t][m] + sum_s X3[s][col] A[t][s]
        float part[4] = {0.f, 0.f, 0.f, 0.f};
        // both column tiles per loaded row fragment: each X1 / A fragment is read
        // once and feeds NCT accumulators
        f32x4 O[NCT][4];
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) O[ct][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh[NCT], fl[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                if constexpr (RP) split_acc<T, SPS>(S[ct][2 * ks], S[ct][2 * ks + 1], fh[ct], fl[ct]);
                else split_acc_plain<T, SPS>(S[ct][2 * ks], S[ct][2 * ks + 1], fh[ct], fl[ct]);
            }
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const frag_t<T> xf = ldfrag(sX1, LDN, 16 * tt, 32 * ks, lane);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) mma2<T, SPS>(O[ct][tt], fh[ct], fl[ct], xf);
            }
        }
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            const float sqt = sq[16 * tt + n16];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) O[ct][tt] *= sqt;
        }
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> vf[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) vf[ct] = ldfragTR<T, LDN, SWX>(sX3, troc, 32 * ks, ccol0 + ccstep * ct);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (32 * ks > 16 * tt + 15) continue;
                const int aw = sizeof(T) == 2 ? 8 * ((lane >> 2) & 1) : 0;
                const frag_t<T> ah = *reinterpret_cast<const frag_t<T> *>(sA + (16 * tt + (lane & 15)) * LDT + ((32 * ks + 8 * (lane >> 4)) ^ aw));
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) mma(O[ct][tt], vf[ct], ah);
                if constexpr (SP) {
                    const frag_t<T> al = *reinterpret_cast<const frag_t<T> *>(sAl + (16 * tt + (lane & 15)) * LDT + ((32 * ks + 8 * (lane >> 4)) ^ aw));
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) mma(O[ct][tt], vf[ct], al);
                }
            }
        }
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                yo[ct][tt] = pack4<T>(O[ct][tt]);
                if constexpr (DQ) {
                    const vec4T qv = qn[4 * ct + tt];
                    part[tt] += O[ct][tt][0] * tof<T>(qv[0]) + O[ct][tt][1] * tof<T>(qv[1]) +
                                O[ct][tt][2] * tof<T>(qv[2]) + O[ct][tt][3] * tof<T>(qv[3]);
                }
            }
        if constexpr (DQ) {
            if (c + 1 < d.nch) issue_q(c + 1);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                part[tt] = sum_rows(part[tt]);
                if (q4 == 0) sred[w * C + 16 * tt + n16] = part[tt];
            }
        }
        sched_fence();
        __syncthreads();  // every wave is done with the score tiles
        put_y();
        sched_fence();

        // state update S = exp2(b63) S + X2^T (exp2(b63 - b) o X3)
        const float gam = fexp2(b63);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < NK; ++i) S[ct][i] *= gam;
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const int s0 = 32 * ks + 8 * q4;
            const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&se[s0]);
            const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&se[s0 + 4]);
            const float ev[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
            frag_t<T> vh[NCT], vl[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
                split_scaled<T, SPD>(ldfragTR<T, LDN, SWX>(sX3, troc, 32 * ks, ccol0 + ccstep * ct), ev, vh[ct], vl[ct]);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> kf = ldfragTR<T, LDN, SWX>(sX2, tro8, 32 * ks, RP ? 32 * (i >> 1) + 4 * (i & 1) : 16 * i);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) mma2b<T, SPD>(S[ct][i], kf, vh[ct], vl[ct]);
            }
        }
    }
    if (d.nch > 0) {
        __syncthreads();
        store_y(d.nch - 1);
    }
    if constexpr (DQ) {
        __syncthreads();
        if (w == 0 && d.nch > 0) {
            float r = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) r += sred[ww * C + lane];
            dgp[(int64_t)((d.nch - 1) * C + lane) * a.sg_l] = r;
        }
    }

    if (a.n_super == 1) {
        if constexpr (!DQ) {
            if (a.S_out) {
                float *dst = a.S_out + d.bh * SS;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int i = 0; i < NK; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            dst[(int64_t)srow(i, r) * D + scol(ct, n16)] = S[ct][i][r];
            }
        } else {
            // <dS_out, S_out> for dg (the state here is S_out^T)
            float p = 0.f;
            if (a.dS_out) {
                const float *ds = a.dS_out + d.bh * SS;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int i = 0; i < NK; ++i) {
                        const f32x4 x = *reinterpret_cast<const f32x4 *>(
                            ds + (int64_t)scol(ct, n16) * D + srow(i, 0));
                        p += x[0] * S[ct][i][0] + x[1] * S[ct][i][1] + x[2] * S[ct][i][2] + x[3] * S[ct][i][3];
                    }
            }
            p = wave_sum(p);
            const int ndot = D * D / 256;
            float *dot = a.wsDot + (int64_t)d.bh * ndot;
            if (lane == 0) dot[w] = p;
            if (w == 0 && lane >= NW && lane < ndot) dot[lane] = 0.f;
        }
    }
}

// ---------------------------------------------------------------------------
// PG: reverse walk over the chunks of a superchunk with the state gradient G
// (dLoss/dS of the state leaving the chunk) in registers:
//   dv^T = exp(b_63 - b_s) G^T K^T + dO^T A^T      (A from Q K^T)
//   dk^T = exp(b_63 - b_s) G V^T   + Q^T dA^T      (dA from dO V^T)
//   G   <- exp(b_63) G + Q^T (exp(b) o dO)          (and its transpose)
//   dg_t = sum_{t' >= t in superchunk} (q.dq - k.dk)_{t'} + <G_{J+1}, S_{J+1}>
// (the last term is the decay gradient carried in from later superchunks).
// The workgroup has two halves of D/(16 NCT) waves.  Wave j of the v-side half
// keeps G[k][v] for its NCT v-tiles (A-operand fragments for dv) and computes
// dv; wave j of the k-side half keeps G^T[v][k] for its NCT k-tiles and
// computes dk and k.dk.  Each half updates only its own orientation, so per
// wave the products, the hi/lo splits and the registers are half of a
// both-orientations walk.  bf16 at d = 128 runs NCT = 2 (8 waves, two per SIMD,
// every K/V/Q/dO fragment read from LDS feeding four MFMAs); the other forms
// NCT = 1.  The v-side half stages q and dO, the k-side half k and v.  LDS
// holds natural tiles only: K and V plain and unswizzled (they meet the G
// fragments split from accumulator pairs: bf16 builds G's rows in the split's
// plain order, see the update; fp32 reorders them with split_acc_plain), Q and
// dO plain and swizzled for the transposing loads of the G updates, where the
// per-token decay goes on the wave's own columns.
template <typename T, int D, int NCT>
__global__ void __launch_bounds__(128 * D / (16 * NCT)) k_bwd_dkv(SegArgs a) {
    constexpr int NJ = D / (16 * NCT), NW = 2 * NJ, NT = 64 * NW, NH = NT / 2, NK = D / 16;
    constexpr int DGW = NJ;  // the wave that finishes dg (the first k-side wave)
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplitScores<T>, SPS = kSplitState<T>, SPD = kSplitDecay<T>;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, plain, swizzled
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];   // plain
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];   // plain
    __shared__ __attribute__((aligned(16))) T sAT[C * LDT];  // A^T[s][t] (hi)
    __shared__ __attribute__((aligned(16))) T sATl[SP ? C * LDT : 8];
    __shared__ __attribute__((aligned(16))) T sdAT[C * LDT]; // dA^T[s][t] (hi)
    __shared__ __attribute__((aligned(16))) T sdATl[SP ? C * LDT : 8];
    __shared__ __attribute__((aligned(16))) float sb[C];   // b_t (log2, chunk-local)
    __shared__ __attribute__((aligned(16))) float se[C];   // exp2(b63 - b_s)
    __shared__ __attribute__((aligned(16))) float sq[C];   // exp2(b_t)
    __shared__ float sred[NJ * C];

    // the wave index through readfirstlane: the compiler then keeps the role and
    // every role-selected pointer in scalar registers
    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool kside = w >= NJ;
    const int j = kside ? w - NJ : w, c0 = 16 * NCT * j, htid = kside ? tid - NH : tid;
    const Decode d = decode(a);
    // score tiles XOR their 16-byte blocks by bit 2 of the row (bf16): the 8-byte
    // accumulator-row writes then spread over twice the banks
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };
    auto ldfrag_a = [&](const T *M, int row0, int k0) {
        return *reinterpret_cast<const frag_t<T> *>(M + (row0 + n16) * LDT + ((k0 + 8 * q4) ^ asw(n16)));
    };
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    // bf16: the rows of G (v-side; of G^T on the k-side) are read into the
    // update's A operands in the order that puts channels 8q..8q+7 of each
    // 32-channel block in lane row q of the accumulator pair (2m, 2m+1), the
    // plain order of the decayed-state product's operand: row r of tile i holds
    // channel grow(i, r), and the pair splits with no lane swaps
    constexpr bool RP = sizeof(T) == 2;
    const LaneOff tro8 = RP ? tr_off8<T, LDN, SWX>(lane) : tro;  // (tr_off8 serves 16-bit tiles only)
    auto grow = [&](int i, int r) { return RP ? 32 * (i >> 1) + 8 * q4 + 4 * (i & 1) + r : 16 * i + 4 * q4 + r; };
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    const T *dO = (const T *)a.dO + xo;
    T *Out = (T *)(kside ? a.dk : a.dv) + xo;
    const int64_t go = d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const float *gp = a.g + go;
    float *dgp = a.dg + go;
    const int64_t SS = (int64_t)D * D;
    const int ndot = D * D / 256;
    // role operands: the B side of the decayed-state product, the own-column
    // transposed tile of the intra-chunk product and of the G update, the score
    // tile, and the shared operand of the G update
    const T *Xs = kside ? sV : sK;
    const T *Own = kside ? sQ : sO;
    const T *Oth = kside ? sO : sQ;
    const T *At = kside ? sdAT : sAT;
    const T *Atl = kside ? sdATl : sATl;

    const float *gsrc = a.n_super == 1 ? (a.dS_out ? a.dS_out + d.bh * SS : nullptr)
                                       : a.wsE + ((int64_t)d.bh * a.n_super + d.J) * SS;
    // v-side: G[k][v] rows 16i.. of the wave's v-tiles; k-side: G^T[v][k] rows of its k-tiles
    f32x4 G[NCT][NK];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int col = c0 + 16 * ct + n16;
            if (!gsrc) {
                G[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};
            } else if (!kside) {
#pragma unroll
                for (int r = 0; r < 4; ++r) G[ct][i][r] = gsrc[(int64_t)grow(i, r) * D + col];
            } else {
                G[ct][i] = *reinterpret_cast<const f32x4 *>(gsrc + (int64_t)col * D + grow(i, 0));
            }
        }
    float carry = 0.f;  // wave DGW: decay gradient carried in from later tokens
    if (w == DGW) {
        const float *dot = a.wsDot + ((int64_t)d.bh * a.n_super + d.J) * ndot;
        carry = wave_sum(lane < ndot ? dot[lane] : 0.f);
    }
    // score tiles read by the dv/dk products but above the diagonal stay zero
    for (int e = tid; e < 512; e += NT) {
        const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
        const int idx = (tile ? (48 + rr) * LDT : (16 + rr) * LDT) + ((tile ? 32 + cc : cc) ^ asw(rr));
        sAT[idx] = cvt<T>(0.f);
        sdAT[idx] = cvt<T>(0.f);
        if constexpr (SP) {
            sATl[idx] = cvt<T>(0.f);
            sdATl[idx] = cvt<T>(0.f);
        }
    }

    // each half loads two tiles (v-side q, dO; k-side k, v) one chunk ahead
    using HT = Tile<T, D, NH>;
    HT t1, t2;
    float gl, rn;
    const int64_t cstep = (int64_t)C * a.sx_l;
    const uint32_t cspan = chunk_span<T, D>(a.sx_l), gspan = (uint32_t)(((C - 1) * a.sg_l + 1) * 4);
    uint32_t toff[HT::RPT];
    HT::offsets(toff, a.sx_l, htid);
    const uint32_t goff = (uint32_t)(lane * a.sg_l * 4);
    const uint32_t tstep = (uint32_t)(16 * a.sx_l * (int64_t)sizeof(T));
    const T *L1 = kside ? K : Q, *L2 = kside ? V : dO;
    auto issue = [&](int c) {
        const int64_t nx = c * cstep;
        t1.load_buf(buf_rsrc(L1 + nx, cspan), toff, 0);
        t2.load_buf(buf_rsrc(L2 + nx, cspan), toff, 0);
    };
    auto issue_g = [&](int c) {
        const int64_t ng = (int64_t)c * C * a.sg_l;
        gl = buf_ld<float>(buf_rsrc(gp + ng, gspan), goff, 0);
        rn = buf_ld<float>(buf_rsrc(dgp + ng, gspan), goff, 0);  // q.dq left in dg by the dq walk
    };
    issue_g(d.nch - 1);
    issue(d.nch - 1);
    float rprev = 0.f;  // wave DGW: q.dq of the chunk whose dg is still pending

    // dg of chunk cp from the k.dk partials in sred (wave DGW)
    auto finish_dg = [&](int cp) {
        float kd = 0.f;
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) kd += sred[jj * C + lane];
        const float suf = wave_incl_suffix(rprev - kd, lane);
        dgp[((int64_t)cp * C + lane) * a.sg_l] = carry + suf;
        carry += lane_value(suf, 0);
    };

    for (int c = d.nch - 1; c >= 0; --c) {
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        const float rc = rn;
        __syncthreads();
        if (!kside) {
            t1.store_swz(sQ, LDN, htid, SWX);
            t2.store_swz(sO, LDN, htid, SWX);
        } else {
            t1.store_swz(sK, LDN, htid, 0);
            t2.store_swz(sV, LDN, htid, 0);
        }
        if (w == NW - 1) {  // the decay tables, from another wave than the dg finish
            sb[lane] = b2;
            se[lane] = fexp2(b63 - b2);
            sq[lane] = fexp2(b2);
        }
        if (c > 0) issue_g(c - 1);
        __syncthreads();
        if (c > 0 && !kside) issue(c - 1);
        // a k-side wave, with one score tile fewer than the v-side waves,
        // finishes the previous chunk's dg beside the scores (walk 0.7% faster
        // than wave 0 doing it in the staging, which every wave waits for)
        if (w == DGW) {
            if (c < d.nch - 1) finish_dg(c + 1);
            rprev = rc;
        }

        // A^T and dA^T on the causal tiles: P[t][s] = sum X[t][ch] Y[s][ch]
        for (int i = w; i < 20; i += NW) {
            const bool isdA = i >= 10;
            int tt, st;
            tri_tile(isdA ? i - 10 : i, tt, st);
            const T *X = isdA ? sO : sQ;
            const T *Yt = isdA ? sV : sK;
            f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                mma(p, ldfrag_swz<T, LDN, SWX>(X, swo, 16 * tt, 32 * ks), ldfrag(Yt, LDN, 16 * st, 32 * ks, lane));
            const int s = 16 * st + n16;
            const float bs = sb[s];
            const f32x4 bt = *reinterpret_cast<const f32x4 *>(&sb[16 * tt + 4 * q4]);
            float v4[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * tt + 4 * q4 + r;
                v4[r] = s <= t ? p[r] * fexp2(bt[r] - bs) : 0.f;
            }
            const int o = s * LDT + ((16 * tt + 4 * q4) ^ asw(s));
            if (isdA) st4_split<T, SP>(&sdAT[o], &sdATl[SP ? o : 0], v4);
            else st4_split<T, SP>(&sAT[o], &sATl[SP ? o : 0], v4);
        }
        __syncthreads();
        if (c > 0 && kside) issue(c - 1);
        // the arbiter favours older waves, so the k-side half (younger, with the
        // k.dk dots on top) finished the products last; it runs them at raised
        // priority (the step measured 0.8% faster, the walk 7%)
        if (kside) __builtin_amdgcn_s_setprio(2);

        // decayed state part: out^T[col][s] += G^T X^T over the wave's 16 NCT columns
        f32x4 DX[NCT][4];
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st) DX[ct][st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> xfr[4];
#pragma unroll
            for (int st = 0; st < 4; ++st) xfr[st] = ldfrag(Xs, LDN, 16 * st, 32 * ks, lane);
            frag_t<T> gh[NCT], glo[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                if constexpr (RP) split_acc<T, SPS>(G[ct][2 * ks], G[ct][2 * ks + 1], gh[ct], glo[ct]);
                else split_acc_plain<T, SPS>(G[ct][2 * ks], G[ct][2 * ks + 1], gh[ct], glo[ct]);
            }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int st = 0; st < 4; ++st) mma2<T, SPS>(DX[ct][st], gh[ct], glo[ct], xfr[st]);
        }
        frag_t<T> of0[NCT], of1[NCT];
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            of0[ct] = ldfragTR<T, LDN, SWX>(Own, tro, 0, c0 + 16 * ct);
            of1[ct] = ldfragTR<T, LDN, SWX>(Own, tro, 32, c0 + 16 * ct);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const float es = se[16 * st + n16];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) DX[ct][st] *= es;
        }
        // intra-chunk part: dv^T += dO^T A^T (v side), dk^T += Q^T dA^T (k side), score
        // tiles zero above the diagonal, over the (st, ks) pairs (0,0) (0,1) (1,0)
        // (1,1) (2,1) (3,1), each pair's fragments read two pairs ahead of its products
        struct AF {
            frag_t<T> h, l;
        };
        auto ld_pair = [&](int st, int ks, AF &f) {
            f.h = ldfrag_a(At, 16 * st, 32 * ks);
            if constexpr (SP) f.l = ldfrag_a(Atl, 16 * st, 32 * ks);
        };
        auto mma_pair = [&](int st, int ks, const AF &f) {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const frag_t<T> &ofk = ks ? of1[ct] : of0[ct];
                mma(DX[ct][st], ofk, f.h);
                if constexpr (SP) mma(DX[ct][st], ofk, f.l);
            }
        };
        {
            AF f0, f1;
            ld_pair(0, 0, f0);
            ld_pair(0, 1, f1);
            sched_fence();
            mma_pair(0, 0, f0);
            ld_pair(1, 0, f0);
            sched_fence();
            mma_pair(0, 1, f1);
            ld_pair(1, 1, f1);
            sched_fence();
            mma_pair(1, 0, f0);
            ld_pair(2, 1, f0);
            sched_fence();
            mma_pair(1, 1, f1);
            ld_pair(3, 1, f1);
            sched_fence();
            mma_pair(2, 1, f0);
            mma_pair(3, 1, f1);
        }
        const rsrc_t ro = buf_rsrc(Out + c * cstep, cspan);
        const uint32_t voff = (uint32_t)((n16 * a.sx_l + c0 + 4 * q4) * (int64_t)sizeof(T));
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st)
                st4_buf<T>(ro, voff, st * tstep + 16 * ct * (uint32_t)sizeof(T), DX[ct][st]);
        if (kside) {  // k.dk partials of this wave's 16 NCT channels
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                float kd = 0.f;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const f32x4 kv = ld4f(&sK[(16 * st + n16) * LDN + c0 + 16 * ct + 4 * q4]);
                    kd += DX[ct][st][0] * kv[0] + DX[ct][st][1] * kv[1] + DX[ct][st][2] * kv[2] + DX[ct][st][3] * kv[3];
                }
                kd = sum_rows(kd);
                if (q4 == 0) sred[j * C + 16 * st + n16] = kd;
            }
        }

        __builtin_amdgcn_s_setprio(0);
        // G <- exp2(b63) G + Q^T (exp2(b) o dO) (v side), G^T <- exp2(b63) G^T + dO^T (exp2(b) o Q) (k side)
        const float gam = fexp2(b63);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < NK; ++i) G[ct][i] *= gam;
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const int t0 = 32 * ks + 8 * q4;
            const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&sq[t0]);
            const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&sq[t0 + 4]);
            const float ev[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
            frag_t<T> oh[NCT], ol[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
                split_scaled<T, SPD>(ldfragTR<T, LDN, SWX>(Own, tro, 32 * ks, c0 + 16 * ct), ev, oh[ct], ol[ct]);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> b = ldfragTR<T, LDN, SWX>(Oth, tro8, 32 * ks, RP ? 32 * (i >> 1) + 4 * (i & 1) : 16 * i);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) mma2b<T, SPD>(G[ct][i], b, oh[ct], ol[ct]);
            }
        }
    }
    __syncthreads();
    if (w == DGW && d.nch > 0) finish_dg(0);
    if (a.n_super == 1 && a.dS_in && !kside) {
        float *dst = a.dS_in + d.bh * SS;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(int64_t)grow(i, r) * D + c0 + 16 * ct + n16] = G[ct][i][r];
    }
}

// PG with the two roles in workgroups of their own (D/16 waves each), the form
// used where the one-workgroup walk above does not fit the LDS (fp32 I/O at
// d = 128: four fp32 tiles and two score tiles need 175 KB).  The v-role
// workgroup keeps G[k][v] and writes dv; the k-role workgroup keeps G^T[v][k]
// and writes dk and dg.  Each stages three tiles (q and dO, plus k or v) and
// its one score tile (A^T or dA^T).  The two workgroups of an item lie 8 apart
// in dispatch order, which puts them on the same XCD (L2) for their second
// read of q and dO.  The k role reads k at its dk elements straight from
// memory for the k.dk dots.  Products and their order are those of k_bwd_dkv.
template <typename T, int D>
__global__ void __launch_bounds__(64 * D / 16) k_bwd_dkv_wg(SegArgs a) {
    constexpr int NW = D / 16, NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr bool SP = kSplitScores<T>, SPS = kSplitState<T>, SPD = kSplitDecay<T>;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, plain, swizzled
    __shared__ __attribute__((aligned(16))) T sX[C * LDN];   // k (v role) or v (k role), plain
    __shared__ __attribute__((aligned(16))) T sAT[C * LDT];  // A^T (v role) or dA^T (k role), hi
    __shared__ __attribute__((aligned(16))) T sATl[SP ? C * LDT : 8];
    __shared__ __attribute__((aligned(16))) float sb[C];   // b_t (log2, chunk-local)
    __shared__ __attribute__((aligned(16))) float se[C];   // exp2(b63 - b_s)
    __shared__ __attribute__((aligned(16))) float sq[C];   // exp2(b_t)
    __shared__ float sred[NW * C];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int blk = (int)blockIdx.x;
    const bool kside = (blk >> 3) & 1;
    const int item = (blk >> 4) * 8 + (blk & 7);
    if (item >= a.B * a.H * a.n_super) return;  // the last group of 8 items is ragged
    const int c0 = 16 * w;
    const Decode d = decode(a, item);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };
    auto ldfrag_a = [&](const T *M, int row0, int k0) {
        return *reinterpret_cast<const frag_t<T> *>(M + (row0 + n16) * LDT + ((k0 + 8 * q4) ^ asw(n16)));
    };
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    const int64_t xo = d.b * a.sx_b + d.h * a.sx_h + d.tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    const T *dO = (const T *)a.dO + xo;
    T *Out = (T *)(kside ? a.dk : a.dv) + xo;
    const int64_t go = d.b * a.sg_b + d.h * a.sg_h + d.tok0 * a.sg_l;
    const float *gp = a.g + go;
    float *dgp = a.dg + go;
    const int64_t SS = (int64_t)D * D;
    const int ndot = D * D / 256;
    // role operands: the own-column transposed tile of the intra-chunk product
    // and of the G update, the shared operand of the G update, and the t side
    // of the score product (A = Q K^T, dA = dO V^T); sX is the other side of
    // the scores and the B side of the decayed-state product
    const T *Own = kside ? sQ : sO;
    const T *Oth = kside ? sO : sQ;
    const T *Xt = kside ? sO : sQ;

    const float *gsrc = a.n_super == 1 ? (a.dS_out ? a.dS_out + d.bh * SS : nullptr)
                                       : a.wsE + ((int64_t)d.bh * a.n_super + d.J) * SS;
    f32x4 G[NK];  // v role: G[k][v] rows 16i.. of v-tile w; k role: G^T[v][k] rows of k-tile w
#pragma unroll
    for (int i = 0; i < NK; ++i) {
        if (!gsrc) {
            G[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        } else if (!kside) {
#pragma unroll
            for (int r = 0; r < 4; ++r) G[i][r] = gsrc[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16];
        } else {
            G[i] = *reinterpret_cast<const f32x4 *>(gsrc + (int64_t)(c0 + n16) * D + 16 * i + 4 * q4);
        }
    }
    float carry = 0.f;  // k role, wave 0: decay gradient carried in from later tokens
    if (kside && w == 0) {
        const float *dot = a.wsDot + ((int64_t)d.bh * a.n_super + d.J) * ndot;
        carry = wave_sum(lane < ndot ? dot[lane] : 0.f);
    }
    // score tile entries read by the products but above the diagonal stay zero
    for (int e = tid; e < 512; e += NT) {
        const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
        const int idx = (tile ? (48 + rr) * LDT : (16 + rr) * LDT) + ((tile ? 32 + cc : cc) ^ asw(rr));
        sAT[idx] = cvt<T>(0.f);
        if constexpr (SP) sATl[idx] = cvt<T>(0.f);
    }

    using HT = Tile<T, D, NT>;
    typedef T vec4T __attribute__((ext_vector_type(4)));
    HT t1, t2, t3;
    float gl, rn = 0.f;
    vec4T kn[4];  // k role: k at this lane's dk elements (tokens 16 st + n16, channels c0 + 4 q4 ..)
    const int64_t cstep = (int64_t)C * a.sx_l;
    const uint32_t cspan = chunk_span<T, D>(a.sx_l), gspan = (uint32_t)(((C - 1) * a.sg_l + 1) * 4);
    uint32_t toff[HT::RPT];
    HT::offsets(toff, a.sx_l, tid);
    const uint32_t goff = (uint32_t)(lane * a.sg_l * 4);
    const uint32_t tstep = (uint32_t)(16 * a.sx_l * (int64_t)sizeof(T));
    const uint32_t voff = (uint32_t)((n16 * a.sx_l + c0 + 4 * q4) * (int64_t)sizeof(T));
    const T *LX = kside ? V : K;
    auto issue_qo = [&](int c) {
        t1.load_buf(buf_rsrc(Q + c * cstep, cspan), toff, 0);
        t2.load_buf(buf_rsrc(dO + c * cstep, cspan), toff, 0);
    };
    auto issue_x = [&](int c) { t3.load_buf(buf_rsrc(LX + c * cstep, cspan), toff, 0); };
    auto issue_k = [&](int c) {
        const rsrc_t rk = buf_rsrc(K + c * cstep, cspan);
#pragma unroll
        for (int st = 0; st < 4; ++st) kn[st] = buf_ld<vec4T>(rk, voff, st * tstep);
    };
    auto issue_g = [&](int c) {
        const int64_t ng = (int64_t)c * C * a.sg_l;
        gl = buf_ld<float>(buf_rsrc(gp + ng, gspan), goff, 0);
        if (kside) rn = buf_ld<float>(buf_rsrc(dgp + ng, gspan), goff, 0);  // q.dq left in dg by the dq walk
    };
    issue_g(d.nch - 1);
    issue_qo(d.nch - 1);
    issue_x(d.nch - 1);
    if (kside) issue_k(d.nch - 1);
    float rprev = 0.f;  // k role, wave 0: q.dq of the chunk whose dg is still pending

    auto finish_dg = [&](int cp) {
        float kd = 0.f;
#pragma unroll
        for (int jj = 0; jj < NW; ++jj) kd += sred[jj * C + lane];
        const float suf = wave_incl_suffix(rprev - kd, lane);
        dgp[((int64_t)cp * C + lane) * a.sg_l] = carry + suf;
        carry += lane_value(suf, 0);
    };

    for (int c = d.nch - 1; c >= 0; --c) {
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        const float rc = rn;
        __syncthreads();
        t1.store_swz(sQ, LDN, tid, SWX);
        t2.store_swz(sO, LDN, tid, SWX);
        t3.store_swz(sX, LDN, tid, 0);
        if (kside && w == 0) {
            if (c < d.nch - 1) finish_dg(c + 1);
            rprev = rc;
        }
        if (w == NW - 1) {  // the decay tables, from another wave than the dg finish
            sb[lane] = b2;
            se[lane] = fexp2(b63 - b2);
            sq[lane] = fexp2(b2);
        }
        if (c > 0) issue_g(c - 1);
        __syncthreads();
        if (c > 0) issue_qo(c - 1);

        // A^T (v role) or dA^T (k role) on the causal tiles: P[t][s] = sum X[t][ch] Y[s][ch]
        for (int i = w; i < 10; i += NW) {
            int tt, st;
            tri_tile(i, tt, st);
            f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                mma(p, ldfrag_swz<T, LDN, SWX>(Xt, swo, 16 * tt, 32 * ks), ldfrag(sX, LDN, 16 * st, 32 * ks, lane));
            const int s = 16 * st + n16;
            const float bs = sb[s];
            const f32x4 bt = *reinterpret_cast<const f32x4 *>(&sb[16 * tt + 4 * q4]);
            float v4[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * tt + 4 * q4 + r;
                v4[r] = s <= t ? p[r] * fexp2(bt[r] - bs) : 0.f;
            }
            const int o = s * LDT + ((16 * tt + 4 * q4) ^ asw(s));
            st4_split<T, SP>(&sAT[o], &sATl[SP ? o : 0], v4);
        }
        __syncthreads();
        if (c > 0) issue_x(c - 1);

        // decayed state part: out^T[col][s] += G^T X^T over the wave's 16 columns
        f32x4 DX[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) DX[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> xfr[4];
#pragma unroll
            for (int st = 0; st < 4; ++st) xfr[st] = ldfrag(sX, LDN, 16 * st, 32 * ks, lane);
            frag_t<T> gh, glo;
            split_acc_plain<T, SPS>(G[2 * ks], G[2 * ks + 1], gh, glo);
#pragma unroll
            for (int st = 0; st < 4; ++st) mma2<T, SPS>(DX[st], gh, glo, xfr[st]);
        }
        const frag_t<T> of0 = ldfragTR<T, LDN, SWX>(Own, tro, 0, c0), of1 = ldfragTR<T, LDN, SWX>(Own, tro, 32, c0);
#pragma unroll
        for (int st = 0; st < 4; ++st) DX[st] *= se[16 * st + n16];
        // intra-chunk part: dv^T += dO^T A^T (v role), dk^T += Q^T dA^T (k role),
        // over the (st, ks) pairs whose score block is not above the diagonal
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int ks = st / 2; ks < C / 32; ++ks) {
                const frag_t<T> &ofk = ks ? of1 : of0;
                mma(DX[st], ofk, ldfrag_a(sAT, 16 * st, 32 * ks));
                if constexpr (SP) mma(DX[st], ofk, ldfrag_a(sATl, 16 * st, 32 * ks));
            }
        const rsrc_t ro = buf_rsrc(Out + c * cstep, cspan);
#pragma unroll
        for (int st = 0; st < 4; ++st) st4_buf<T>(ro, voff, st * tstep, DX[st]);
        if (kside) {  // k.dk partials of this wave's 16 channels, then the next chunk's k
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                float kd = 0.f;
#pragma unroll
                for (int r = 0; r < 4; ++r) kd += DX[st][r] * tof<T>(kn[st][r]);
                kd = sum_rows(kd);
                if (q4 == 0) sred[w * C + 16 * st + n16] = kd;
            }
            if (c > 0) issue_k(c - 1);
        }

        // G <- exp2(b63) G + Q^T (exp2(b) o dO) (v role), G^T <- exp2(b63) G^T + dO^T (exp2(b) o Q) (k role)
        const float gam = fexp2(b63);
#pragma unroll
        for (int i = 0; i < NK; ++i) G[i] *= gam;
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const int t0 = 32 * ks + 8 * q4;
            const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&sq[t0]);
            const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&sq[t0 + 4]);
            const float ev[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
            frag_t<T> oh, ol;
            split_scaled<T, SPD>(ldfragTR<T, LDN, SWX>(Own, tro, 32 * ks, c0), ev, oh, ol);
#pragma unroll
            for (int i = 0; i < NK; ++i) mma2b<T, SPD>(G[i], ldfragTR<T, LDN, SWX>(Oth, tro, 32 * ks, 16 * i), oh, ol);
        }
    }
    __syncthreads();
    if (kside && w == 0 && d.nch > 0) finish_dg(0);
    if (a.n_super == 1 && a.dS_in && !kside) {
        float *dst = a.dS_in + d.bh * SS;
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = G[i][r];
    }
}

// Boundary state of an empty segment: dst = src, or zero when src is NULL.
__global__ void __launch_bounds__(SCAN_NT) k_state_copy(const float *src, float *dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * SCAN_NT + threadIdx.x;
    if (i < n) dst[i] = src ? src[i] : 0.f;
}

// ---------------------------------------------------------------------------
// launchers
template <typename T, int D>
static hipError_t launch_td(int kind, const SegArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((unsigned)((int64_t)a.B * a.H * a.n_super));
    constexpr int NTP = 64 * D / (16 * SF_NCT_PREP);
    constexpr int NTW = 64 * D / (16 * SF_NCT_WALK);
    switch (kind) {
    case SF_K_FWD_PREP: hipExtLaunchKernelGGL((k_prep<T, D, SF_NCT_PREP, false>), grid, dim3(NTP), 0, s, e0, e1, 0, a); break;
    case SF_K_FWD_OUT:
        // a launch that would leave half the CUs idle splits the state's columns
        // over two workgroups per item (scan-bound workload: 5.15 -> 4.98 ms per
        // step; at one item per CU the split measured slower)
        if (sizeof(T) == 2 && D == 128 && 2 * (int64_t)grid.x <= (int64_t)a.n_cu) {
            hipExtLaunchKernelGGL((k_walk<T, D, 1, false, 2>), dim3((grid.x + 7) / 8 * 16), dim3(64 * D / 32), 0, s, e0,
                                  e1, 0, a);
        } else {
            hipExtLaunchKernelGGL((k_walk<T, D, SF_NCT_WALK, false>), grid, dim3(NTW), 0, s, e0, e1, 0, a);
        }
        break;
    case SF_K_BWD_PREP:  // the replay of D_J (the forward's prep), skipped for kept states, then E_J
        if (!a.ckpt)
            hipExtLaunchKernelGGL((k_prep_bwd<T, D, SF_NCT_PREP>), dim3(2 * grid.x), dim3(NTP), 0, s, e0, e1, 0, a);
        else
            hipExtLaunchKernelGGL((k_prep<T, D, SF_NCT_PREP, true>), grid, dim3(NTP), 0, s, e0, e1, 0, a);
        break;
    case SF_K_BWD_DQ: hipExtLaunchKernelGGL((k_walk<T, D, SF_NCT_WALK, true>), grid, dim3(NTW), 0, s, e0, e1, 0, a); break;
    case SF_K_BWD_DKV:
        if constexpr (sizeof(T) == 4 && D == 128) {  // two workgroups per item, 8 apart in dispatch order
            const int64_t items = (int64_t)a.B * a.H * a.n_super;
            hipExtLaunchKernelGGL((k_bwd_dkv_wg<T, D>), dim3((unsigned)((items + 7) / 8 * 16)), dim3(64 * D / 16), 0, s,
                                  e0, e1, 0, a);
        } else {
            constexpr int NCT = sizeof(T) == 2 && D == 128 ? SF_NCT_DKV : 1;
            hipExtLaunchKernelGGL((k_bwd_dkv<T, D, NCT>), grid, dim3(128 * D / (16 * NCT)), 0, s, e0, e1, 0, a);
        }
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_kernel(int kind, int io, int D, const SegArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (kind == SF_K_SCAN) {
        const dim3 grid((unsigned)((int64_t)a.B * a.H * (D * D / 1024)));
        if (a.vec) {
            if (a.wsE) hipExtLaunchKernelGGL((k_scan<true, true>), grid, dim3(SCAN_NT), 0, s, e0, e1, 0, a, D);
            else hipExtLaunchKernelGGL((k_scan<false, true>), grid, dim3(SCAN_NT), 0, s, e0, e1, 0, a, D);
        } else {
            if (a.wsE) hipExtLaunchKernelGGL((k_scan<true, false>), grid, dim3(SCAN_NT), 0, s, e0, e1, 0, a, D);
            else hipExtLaunchKernelGGL((k_scan<false, false>), grid, dim3(SCAN_NT), 0, s, e0, e1, 0, a, D);
        }
        return hipGetLastError();
    }
    if (a.vec) return launch_kernel_vg(kind, io, D, a, s, e0, e1);
    if (io == SF_BF16 && D == 128) return launch_td<__bf16, 128>(kind, a, s, e0, e1);
    if (io == SF_BF16 && D == 64) return launch_td<__bf16, 64>(kind, a, s, e0, e1);
    if (io == SF_F32 && D == 64) return launch_td<float, 64>(kind, a, s, e0, e1);
    if (io == SF_F32 && D == 128) return launch_td<float, 128>(kind, a, s, e0, e1);
    return hipErrorInvalidValue;
}

hipError_t launch_state_copy(const float *src, float *dst, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_state_copy, dim3((unsigned)((n + SCAN_NT - 1) / SCAN_NT)), dim3(SCAN_NT), 0, s, src, dst,
                       n);
    return hipGetLastError();
}

}  // namespace sf
