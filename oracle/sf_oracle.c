/*
 * sf_oracle.c -- fp64 CPU oracle for the segmented gated linear recurrence.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this library.  It shares no code,
 * header, table or helper with the HIP library; the product path never
 * calls it.
 *
 * What it computes (paper, Sec. 2.1 "Modern Linear Recurrence", Eq. 1, with
 * the scalar-identity transition F_t = a_t I of Mamba-2/3 and the per-key-
 * channel diagonal transition read for GLA; state stored as S in R^{Dk x Dv},
 * the transpose of the paper's S in R^{Dv x Dk}):
 *
 *     S_t = a_t o S_{t-1} + k_t v_t^T,     o_t = S_t^T q_t,     a_t = exp(g_t)
 *
 * token by token, with S_{-1} = S_in (zero when absent; the paper's S_0 = 0).
 * "a_t o S" is a_t * S for a scalar gate and diag(a_t) S for a vector gate.
 *
 * The backward pass is the exact reverse-mode derivative of
 *     Loss = sum_t <dO_t, o_t> + <dS_out, S_out>
 * written out by hand (Sec. 3.1 "Backward Computation": the segment backward
 * consumes the output-boundary gradient dS_out and produces dS_in):
 *
 *     G <- dS_out
 *     for t = L-1 .. 0:
 *         G     <- G + q_t dO_t^T             (G is now dLoss/dS_t)
 *         dq_t   = S_t dO_t
 *         dk_t   = G v_t
 *         dv_t   = G^T k_t
 *         dg_t   = a_t <G, S_{t-1}>           (vector gate: per key row c)
 *         G     <- a_t o G
 *     dS_in = G
 *
 * The states S_t needed in reverse order are recomputed forward from
 * checkpoints taken every BLK tokens; the recurrence is never inverted.
 *
 * Layouts (double, contiguous):
 *   q, k, dq, dk : [B][L][H][Dk]       v, dO, o, dv : [B][L][H][Dv]
 *   g, dg        : [B][L][H]  (scalar gate)  or  [B][L][H][Dk] (vector gate)
 *   states       : [B][H][Dk][Dv]
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int B, H, Dk, Dv, vec;
    long L;
} dims_t;

static inline long xi(const dims_t *d, int b, long t, int h, int D) {
    return (((long)b * d->L + t) * d->H + h) * (long)D;
}
static inline long gi(const dims_t *d, int b, long t, int h) {
    return xi(d, b, t, h, d->vec ? d->Dk : 1);
}
static inline long si(const dims_t *d, int b, int h) {
    return ((long)b * d->H + h) * (long)d->Dk * d->Dv;
}

/* S <- a o S + k v^T for one token (Eq. 1, update rule). */
static void update(const dims_t *d, double *S, const double *g, const double *k,
                   const double *v) {
    for (int c = 0; c < d->Dk; ++c) {
        double a = exp(d->vec ? g[c] : g[0]);
        double *row = S + (long)c * d->Dv;
        for (int j = 0; j < d->Dv; ++j) row[j] = a * row[j] + k[c] * v[j];
    }
}

/* o = S^T q (Eq. 1, query rule). */
static void query(const dims_t *d, const double *S, const double *q, double *o) {
    for (int j = 0; j < d->Dv; ++j) o[j] = 0.0;
    for (int c = 0; c < d->Dk; ++c) {
        const double *row = S + (long)c * d->Dv;
        for (int j = 0; j < d->Dv; ++j) o[j] += row[j] * q[c];
    }
}

/*
 * Forward.  S_in may be NULL (zero state).  If n_snap > 0, snap receives the
 * state after snap_pos[p] tokens, layout [n_snap][B][H][Dk][Dv]; snap_pos must
 * be in [0, L].  Returns 0 on success, -1 on allocation failure, -2 on bad
 * arguments.
 */
int sfo_forward(int B, int H, int Dk, int Dv, long L, int vector_gate,
                const double *q, const double *k, const double *v, const double *g,
                const double *S_in, double *o, double *S_out,
                int n_snap, const long *snap_pos, double *snap, int n_threads) {
    if (B < 1 || H < 1 || Dk < 1 || Dv < 1 || L < 0) return -2;
    if (L > 0 && (!q || !k || !v || !g || !o)) return -2;
    if (!S_out || (n_snap > 0 && (!snap_pos || !snap))) return -2;
    for (int p = 0; p < n_snap; ++p)
        if (snap_pos[p] < 0 || snap_pos[p] > L) return -2;
    dims_t d = {B, H, Dk, Dv, vector_gate ? 1 : 0, L};
    const long SS = (long)Dk * Dv;
    const long nstate = (long)B * H * SS;
    int err = 0;
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#endif
#pragma omp parallel for schedule(dynamic, 1)
    for (int task = 0; task < B * H; ++task) {
        int b = task / H, h = task % H;
        double *S = (double *)malloc(sizeof(double) * SS);
        if (!S) {
#pragma omp atomic write
            err = -1;
            continue;
        }
        if (S_in) memcpy(S, S_in + si(&d, b, h), sizeof(double) * SS);
        else memset(S, 0, sizeof(double) * SS);
        for (int p = 0; p < n_snap; ++p)
            if (snap_pos[p] == 0) memcpy(snap + p * nstate + si(&d, b, h), S, sizeof(double) * SS);
        for (long t = 0; t < L; ++t) {
            update(&d, S, g + gi(&d, b, t, h), k + xi(&d, b, t, h, Dk), v + xi(&d, b, t, h, Dv));
            query(&d, S, q + xi(&d, b, t, h, Dk), o + xi(&d, b, t, h, Dv));
            for (int p = 0; p < n_snap; ++p)
                if (snap_pos[p] == t + 1)
                    memcpy(snap + p * nstate + si(&d, b, h), S, sizeof(double) * SS);
        }
        memcpy(S_out + si(&d, b, h), S, sizeof(double) * SS);
        free(S);
    }
    return err;
}

/*
 * Backward.  S_in and dS_out may be NULL (zero).  Returns 0 on success.
 */
int sfo_backward(int B, int H, int Dk, int Dv, long L, int vector_gate,
                 const double *q, const double *k, const double *v, const double *g,
                 const double *S_in, const double *dO, const double *dS_out,
                 double *dq, double *dk, double *dv, double *dg, double *dS_in,
                 int n_threads) {
    if (B < 1 || H < 1 || Dk < 1 || Dv < 1 || L < 0) return -2;
    if (L > 0 && (!q || !k || !v || !g || !dO || !dq || !dk || !dv || !dg)) return -2;
    if (!dS_in) return -2;
    dims_t d = {B, H, Dk, Dv, vector_gate ? 1 : 0, L};
    const long SS = (long)Dk * Dv;
    long blk = (long)sqrt((double)(L > 0 ? L : 1));
    if (blk < 16) blk = 16;
    const long nblk = L > 0 ? (L + blk - 1) / blk : 0;
    int err = 0;
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#endif
#pragma omp parallel for schedule(dynamic, 1)
    for (int task = 0; task < B * H; ++task) {
        int b = task / H, h = task % H;
        /* ckpt[i] = state entering block i; Sb[j] = state after j tokens of the block */
        double *ckpt = (double *)malloc(sizeof(double) * SS * (nblk > 0 ? nblk : 1));
        double *Sb = (double *)malloc(sizeof(double) * SS * (blk + 1));
        double *G = (double *)malloc(sizeof(double) * SS);
        if (!ckpt || !Sb || !G) {
            free(ckpt); free(Sb); free(G);
#pragma omp atomic write
            err = -1;
            continue;
        }
        /* forward sweep: checkpoints only */
        double *S = Sb;
        if (S_in) memcpy(S, S_in + si(&d, b, h), sizeof(double) * SS);
        else memset(S, 0, sizeof(double) * SS);
        for (long i = 0; i < nblk; ++i) {
            memcpy(ckpt + i * SS, S, sizeof(double) * SS);
            long t1 = (i + 1) * blk < L ? (i + 1) * blk : L;
            for (long t = i * blk; t < t1; ++t)
                update(&d, S, g + gi(&d, b, t, h), k + xi(&d, b, t, h, Dk), v + xi(&d, b, t, h, Dv));
        }
        /* reverse sweep */
        if (dS_out) memcpy(G, dS_out + si(&d, b, h), sizeof(double) * SS);
        else memset(G, 0, sizeof(double) * SS);
        for (long i = nblk - 1; i >= 0; --i) {
            long t0 = i * blk;
            long t1 = (i + 1) * blk < L ? (i + 1) * blk : L;
            memcpy(Sb, ckpt + i * SS, sizeof(double) * SS);
            for (long t = t0; t < t1; ++t) {
                memcpy(Sb + (t - t0 + 1) * SS, Sb + (t - t0) * SS, sizeof(double) * SS);
                update(&d, Sb + (t - t0 + 1) * SS, g + gi(&d, b, t, h),
                       k + xi(&d, b, t, h, Dk), v + xi(&d, b, t, h, Dv));
            }
            for (long t = t1 - 1; t >= t0; --t) {
                const double *St = Sb + (t - t0 + 1) * SS;
                const double *Sp = Sb + (t - t0) * SS;
                const double *qt = q + xi(&d, b, t, h, Dk);
                const double *kt = k + xi(&d, b, t, h, Dk);
                const double *vt = v + xi(&d, b, t, h, Dv);
                const double *dot = dO + xi(&d, b, t, h, Dv);
                const double *gt = g + gi(&d, b, t, h);
                double *dqt = dq + xi(&d, b, t, h, Dk);
                double *dkt = dk + xi(&d, b, t, h, Dk);
                double *dvt = dv + xi(&d, b, t, h, Dv);
                double *dgt = dg + gi(&d, b, t, h);
                /* G <- G + q_t dO_t^T */
                for (int c = 0; c < Dk; ++c)
                    for (int j = 0; j < Dv; ++j) G[(long)c * Dv + j] += qt[c] * dot[j];
                /* dq_t = S_t dO_t ; dk_t = G v_t */
                for (int c = 0; c < Dk; ++c) {
                    double sq = 0.0, sk = 0.0;
                    for (int j = 0; j < Dv; ++j) {
                        sq += St[(long)c * Dv + j] * dot[j];
                        sk += G[(long)c * Dv + j] * vt[j];
                    }
                    dqt[c] = sq;
                    dkt[c] = sk;
                }
                /* dv_t = G^T k_t */
                for (int j = 0; j < Dv; ++j) dvt[j] = 0.0;
                for (int c = 0; c < Dk; ++c)
                    for (int j = 0; j < Dv; ++j) dvt[j] += G[(long)c * Dv + j] * kt[c];
                /* dg_t = a_t <G, S_{t-1}> (per key row for the vector gate) */
                if (d.vec) {
                    for (int c = 0; c < Dk; ++c) {
                        double s = 0.0;
                        for (int j = 0; j < Dv; ++j) s += G[(long)c * Dv + j] * Sp[(long)c * Dv + j];
                        dgt[c] = exp(gt[c]) * s;
                    }
                } else {
                    double s = 0.0;
                    for (long e = 0; e < SS; ++e) s += G[e] * Sp[e];
                    dgt[0] = exp(gt[0]) * s;
                }
                /* G <- a_t o G */
                for (int c = 0; c < Dk; ++c) {
                    double a = exp(d.vec ? gt[c] : gt[0]);
                    for (int j = 0; j < Dv; ++j) G[(long)c * Dv + j] *= a;
                }
            }
        }
        memcpy(dS_in + si(&d, b, h), G, sizeof(double) * SS);
        free(ckpt); free(Sb); free(G);
    }
    return err;
}

int sfo_version(void) { return 1; }
