/*
 * gdn_oracle.c -- fp64 CPU oracle for the gated delta rule (GDN).
 *
 * TEST INFRASTRUCTURE ONLY (same rules as sf_oracle.c: tests/, smoke() and
 * bench.py's cpu_baseline leg may load it; it shares nothing with the HIP
 * library).
 *
 * The paper's recurrence S_t = S_{t-1} F_t + v_t k_t^T (Sec. 2.1) with the
 * scalar-plus-low-rank transition of Gated DeltaNet, F_t = a_t (I - beta_t
 * k_t k_t^T), and the write scaled by beta_t as in GDN.  State stored as
 * S in R^{Dk x Dv} (the transpose of the paper's), so per token:
 *
 *     P   = a_t S_{t-1}                       (decay, a_t = exp(g_t))
 *     u_t = beta_t (v_t - P^T k_t)            (the corrected value, V^new)
 *     S_t = P + k_t u_t^T                     (= a_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T)
 *     o_t = S_t^T q_t
 * u_t is the delta rule's corrected value (the V^new that the paper's ST
 * step returns beside the state); gdo_forward can return it.
 *
 * Backward of Loss = sum_t <dO_t, o_t> + <dS_out, S_out>, by hand, per token
 * in reverse with G = dLoss/dS_t:
 *     G    += q_t dO_t^T;     dq_t = S_t dO_t
 *     dk_t  = G u_t;          du   = G^T k_t
 *     dbeta_t = <du, v_t - P^T k_t>;  dv_t = beta_t du
 *     dP    = G - beta_t k_t du^T;    dk_t -= beta_t P du
 *     dg_t  = a_t <dP, S_{t-1}>;      G <- a_t dP
 *     dS_in = G after the first token.
 * States are replayed from checkpoints every ~sqrt(L) tokens; the recurrence
 * is never inverted.
 *
 * Layouts (double, contiguous): q, k: [B][L][H][Dk]; v, o, u_out: [B][L][H][Dv];
 * g, beta: [B][L][H]; states [B][H][Dk][Dv].
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int B, H, Dk, Dv;
    long L;
} gdims_t;

static inline long gx(const gdims_t *d, int b, long t, int h, int D) { return (((long)b * d->L + t) * d->H + h) * (long)D; }
static inline long gs(const gdims_t *d, int b, long t, int h) { return ((long)b * d->L + t) * d->H + h; }
static inline long gst(const gdims_t *d, int b, int h) { return ((long)b * d->H + h) * (long)d->Dk * d->Dv; }

/* one token: S (S_{t-1} in, S_t out); u receives u_t */
static void gdn_step(const gdims_t *d, double *S, double g, double beta, const double *k, const double *v,
                     double *u) {
    const double a = exp(g);
    for (long e = 0; e < (long)d->Dk * d->Dv; ++e) S[e] *= a;
    for (int j = 0; j < d->Dv; ++j) {
        double w = 0.0;
        for (int c = 0; c < d->Dk; ++c) w += S[(long)c * d->Dv + j] * k[c];
        u[j] = beta * (v[j] - w);
    }
    for (int c = 0; c < d->Dk; ++c)
        for (int j = 0; j < d->Dv; ++j) S[(long)c * d->Dv + j] += k[c] * u[j];
}

int gdo_forward(int B, int H, int Dk, int Dv, long L, const double *q, const double *k, const double *v,
                const double *g, const double *beta, const double *S_in, double *o, double *S_out, double *u_out,
                int n_threads) {
    if (B < 1 || H < 1 || Dk < 1 || Dv < 1 || L < 0 || !S_out) return -2;
    if (L > 0 && (!q || !k || !v || !g || !beta || !o)) return -2;
    gdims_t d = {B, H, Dk, Dv, L};
    const long SS = (long)Dk * Dv;
    int err = 0;
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#endif
#pragma omp parallel for schedule(dynamic, 1)
    for (int task = 0; task < B * H; ++task) {
        int b = task / H, h = task % H;
        double *S = (double *)malloc(sizeof(double) * SS);
        double *u = (double *)malloc(sizeof(double) * Dv);
        if (!S || !u) {
            free(S); free(u);
#pragma omp atomic write
            err = -1;
            continue;
        }
        if (S_in) memcpy(S, S_in + gst(&d, b, h), sizeof(double) * SS);
        else memset(S, 0, sizeof(double) * SS);
        for (long t = 0; t < L; ++t) {
            gdn_step(&d, S, g[gs(&d, b, t, h)], beta[gs(&d, b, t, h)], k + gx(&d, b, t, h, Dk), v + gx(&d, b, t, h, Dv), u);
            if (u_out) memcpy(u_out + gx(&d, b, t, h, Dv), u, sizeof(double) * Dv);
            const double *qt = q + gx(&d, b, t, h, Dk);
            double *ot = o + gx(&d, b, t, h, Dv);
            for (int j = 0; j < Dv; ++j) {
                double s = 0.0;
                for (int c = 0; c < Dk; ++c) s += S[(long)c * Dv + j] * qt[c];
                ot[j] = s;
            }
        }
        memcpy(S_out + gst(&d, b, h), S, sizeof(double) * SS);
        free(S); free(u);
    }
    return err;
}

int gdo_backward(int B, int H, int Dk, int Dv, long L, const double *q, const double *k, const double *v,
                 const double *g, const double *beta, const double *S_in, const double *dO, const double *dS_out,
                 double *dq, double *dk, double *dv, double *dg, double *dbeta, double *dS_in, int n_threads) {
    if (B < 1 || H < 1 || Dk < 1 || Dv < 1 || L < 0 || !dS_in) return -2;
    if (L > 0 && (!q || !k || !v || !g || !beta || !dO || !dq || !dk || !dv || !dg || !dbeta)) return -2;
    gdims_t d = {B, H, Dk, Dv, L};
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
        double *ckpt = (double *)malloc(sizeof(double) * SS * (nblk > 0 ? nblk : 1));
        double *Sb = (double *)malloc(sizeof(double) * SS * (blk + 1));
        double *G = (double *)malloc(sizeof(double) * SS);
        double *P = (double *)malloc(sizeof(double) * SS);
        double *u = (double *)malloc(sizeof(double) * Dv);
        double *r = (double *)malloc(sizeof(double) * Dv);
        double *du = (double *)malloc(sizeof(double) * Dv);
        if (!ckpt || !Sb || !G || !P || !u || !r || !du) {
            free(ckpt); free(Sb); free(G); free(P); free(u); free(r); free(du);
#pragma omp atomic write
            err = -1;
            continue;
        }
        double *S = Sb;
        if (S_in) memcpy(S, S_in + gst(&d, b, h), sizeof(double) * SS);
        else memset(S, 0, sizeof(double) * SS);
        for (long i = 0; i < nblk; ++i) {
            memcpy(ckpt + i * SS, S, sizeof(double) * SS);
            long t1 = (i + 1) * blk < L ? (i + 1) * blk : L;
            for (long t = i * blk; t < t1; ++t)
                gdn_step(&d, S, g[gs(&d, b, t, h)], beta[gs(&d, b, t, h)], k + gx(&d, b, t, h, Dk),
                         v + gx(&d, b, t, h, Dv), u);
        }
        if (dS_out) memcpy(G, dS_out + gst(&d, b, h), sizeof(double) * SS);
        else memset(G, 0, sizeof(double) * SS);
        for (long i = nblk - 1; i >= 0; --i) {
            long t0 = i * blk, t1 = (i + 1) * blk < L ? (i + 1) * blk : L;
            memcpy(Sb, ckpt + i * SS, sizeof(double) * SS);
            for (long t = t0; t < t1; ++t) {
                memcpy(Sb + (t - t0 + 1) * SS, Sb + (t - t0) * SS, sizeof(double) * SS);
                gdn_step(&d, Sb + (t - t0 + 1) * SS, g[gs(&d, b, t, h)], beta[gs(&d, b, t, h)],
                         k + gx(&d, b, t, h, Dk), v + gx(&d, b, t, h, Dv), u);
            }
            for (long t = t1 - 1; t >= t0; --t) {
                const double *St = Sb + (t - t0 + 1) * SS, *Sp = Sb + (t - t0) * SS;
                const double *qt = q + gx(&d, b, t, h, Dk), *kt = k + gx(&d, b, t, h, Dk);
                const double *vt = v + gx(&d, b, t, h, Dv), *dot = dO + gx(&d, b, t, h, Dv);
                const double a = exp(g[gs(&d, b, t, h)]), bt = beta[gs(&d, b, t, h)];
                double *dqt = dq + gx(&d, b, t, h, Dk), *dkt = dk + gx(&d, b, t, h, Dk);
                double *dvt = dv + gx(&d, b, t, h, Dv);
                /* forward quantities of this token: P = a S_{t-1}, r = v - P^T k, u = beta r */
                for (long e = 0; e < SS; ++e) P[e] = a * Sp[e];
                for (int j = 0; j < Dv; ++j) {
                    double w = 0.0;
                    for (int c = 0; c < Dk; ++c) w += P[(long)c * Dv + j] * kt[c];
                    r[j] = vt[j] - w;
                    u[j] = bt * r[j];
                }
                /* G += q dO^T ; dq = S_t dO */
                for (int c = 0; c < Dk; ++c)
                    for (int j = 0; j < Dv; ++j) G[(long)c * Dv + j] += qt[c] * dot[j];
                for (int c = 0; c < Dk; ++c) {
                    double s = 0.0;
                    for (int j = 0; j < Dv; ++j) s += St[(long)c * Dv + j] * dot[j];
                    dqt[c] = s;
                }
                /* S_t = P + k u^T: dk = G u, du = G^T k */
                for (int c = 0; c < Dk; ++c) {
                    double s = 0.0;
                    for (int j = 0; j < Dv; ++j) s += G[(long)c * Dv + j] * u[j];
                    dkt[c] = s;
                }
                for (int j = 0; j < Dv; ++j) {
                    double s = 0.0;
                    for (int c = 0; c < Dk; ++c) s += G[(long)c * Dv + j] * kt[c];
                    du[j] = s;
                }
                /* u = beta (v - P^T k) */
                double db = 0.0;
                for (int j = 0; j < Dv; ++j) {
                    db += du[j] * r[j];
                    dvt[j] = bt * du[j];
                }
                dbeta[gs(&d, b, t, h)] = db;
                /* dP = G - beta k du^T ; dk -= beta P du */
                for (int c = 0; c < Dk; ++c) {
                    double s = 0.0;
                    for (int j = 0; j < Dv; ++j) s += P[(long)c * Dv + j] * du[j];
                    dkt[c] -= bt * s;
                }
                for (int c = 0; c < Dk; ++c)
                    for (int j = 0; j < Dv; ++j) G[(long)c * Dv + j] -= bt * kt[c] * du[j];
                /* P = a S_{t-1}: dg = a <dP, S_{t-1}>, G <- a dP */
                double s = 0.0;
                for (long e = 0; e < SS; ++e) s += G[e] * Sp[e];
                dg[gs(&d, b, t, h)] = a * s;
                for (long e = 0; e < SS; ++e) G[e] *= a;
            }
        }
        memcpy(dS_in + gst(&d, b, h), G, sizeof(double) * SS);
        free(ckpt); free(Sb); free(G); free(P); free(u); free(r); free(du);
    }
    return err;
}
