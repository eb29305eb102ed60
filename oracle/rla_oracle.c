/*
 * Reference (oracle) implementation of the RLA and RDN sequence-mixing
 * operators, in plain fp64 C, token by token.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the independent CPU definition the
 * GPU library is checked against.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg load it; the GPU library never links,
 * includes or calls it, and it shares no code with the GPU kernels.
 *
 * What it computes (paper: "Enhancing linear attention with residual
 * learning", Sec. 3.4 "Final Formulations", the two boxed recurrences):
 *
 *   x_t = v_t - S_{t-1} k_t                         residual before clipping
 *   r_t = Clip_[-c,c](x_t)                          Sec. 3.3, elementwise
 *   RDN:  R_t = aR_t R_{t-1} (I - g_t k_t k_t^T) + g_t r_t k_t^T
 *         S_t = aS_t S_{t-1} (I - b_t k_t k_t^T) + b_t v_t k_t^T
 *   RLA:  R_t = aR_t R_{t-1} + g_t r_t k_t^T
 *         S_t = aS_t S_{t-1} + b_t v_t k_t^T
 *   o_t = aS_t S_{t-1} q_t + g_t R_t q_t            (old S, new R)
 *
 * The paper uses one decay alpha_t for both states; here the decay of S (aS)
 * and of R (aR) are separate arguments, and aR == aS recovers the paper.
 * g is the correction factor gamma of Sec. 3.2, b is the write strength beta.
 *
 * Storage convention (shared with the GPU library's C ABI, not with its code):
 *   q, k      [ntok][H][dk]       v, o      [ntok][H][dv]
 *   gates     [ntok][H]
 *   states    [N][H][dk][dv]      element (i, j) holds the paper's S[j][i],
 *                                 i.e. the state is stored transposed
 *   cu_seqlens int64 [N+1]        sequence n covers tokens [cu[n], cu[n+1])
 *   clip c < 0 is read as "no clipping" (c = +infinity).
 *
 * The backward pass is the adjoint of the recurrence above (derived by hand:
 * the paper gives only the forward), run in reverse over each sequence with
 * the forward states recomputed from checkpoints taken every CKPT tokens.
 * Its derivation, per token, in the paper's orientation:
 *   output:   dS_{t-1} += aS do q^T ;  dR_t += g do q^T ;
 *             dq += aS S_{t-1}^T do + g R_t^T do ;
 *             daS += do.(S_{t-1} q) ;  dg += do.(R_t q)
 *   R update: z = dR_t k ;  dr = g z ;  dR_{t-1} = aR dR_t (I - g k k^T) ;
 *             daR += <dR_t, R_{t-1}(I - g k k^T)> ;  dg += z.(r - aR R_{t-1}k) ;
 *             dk += -aR g (R_{t-1}^T z + dR_t^T R_{t-1} k) + g dR_t^T r
 *   clip:     dx = [|x| <= c] * dr ;  dv += dx ;  dS_{t-1} -= dx k^T ;
 *             dk -= S_{t-1}^T dx
 *   S update: w = dS_t k ;  dS_{t-1} += aS dS_t (I - b k k^T) ;
 *             daS += <dS_t, S_{t-1}(I - b k k^T)> ;  db += w.(v - aS S_{t-1}k) ;
 *             dv += b w ;  dk += -aS b (S_{t-1}^T w + dS_t^T S_{t-1} k) + b dS_t^T v
 * (RLA drops every term that comes from the (I - . k k^T) factors.)
 * The clip's derivative is taken as 1 on the closed interval [-c, c].
 *
 * Variants (bits of `variant` above bit 0, which selects RDN over RLA):
 *   ORC_TANH     r_t = c tanh(x_t / c): the negative gradient of the scaled
 *                log-cosh loss c^2 log cosh((v - v_hat) / c), the robust
 *                alternative to the clipped residual of App. B (c = 1 is the
 *                paper's plain tanh; c = inf gives r = x, c = 0 gives r = 0).
 *                Its derivative 1 - tanh^2(x / c) replaces the clip mask.
 *   ORC_UNGATED  o_t = S_{t-1} q_t + R_t q_t, the ungated output combination
 *                of the ablation in Sec. 4.3.
 *   ORC_DECAYED  x_t = v_t - aS_t S_{t-1} k_t, the residual of the decayed
 *                prediction (the prediction of Table 1's gated rows) in place
 *                of the boxed v_t - S_{t-1} k_t.
 * Backward with the variants: the output adjoint loses its aS and g factors
 * (UNGATED); dx = phi'(x) dr with phi' the derivative of the residual
 * function (TANH); the residual's adjoint carries the factor aS and adds
 * daS -= dx.(S_{t-1} k) (DECAYED).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_RLA 0
#define ORC_RDN 1
#define ORC_TANH 2
#define ORC_UNGATED 4
#define ORC_DECAYED 8
#define CKPT 64

static double clip_value(double x, double c) {
    if (c < 0.0) return x;            /* no clipping */
    if (x > c) return c;
    if (x < -c) return -c;
    return x;
}

static int clip_passes(double x, double c) {
    if (c < 0.0) return 1;
    return (x >= -c && x <= c) ? 1 : 0;
}

/* residual function r = phi(x) and its derivative phi'(x) */
static double resid_value(int variant, double x, double c) {
    if (!(variant & ORC_TANH)) return clip_value(x, c);
    if (c < 0.0) return x;
    if (c == 0.0) return 0.0;
    return c * tanh(x / c);
}

static double resid_slope(int variant, double x, double c) {
    double th;
    if (!(variant & ORC_TANH)) return clip_passes(x, c) ? 1.0 : 0.0;
    if (c < 0.0) return 1.0;
    if (c == 0.0) return 0.0;
    th = tanh(x / c);
    return 1.0 - th * th;
}

/* Scratch for one (sequence, head) pair. */
typedef struct {
    double *Sk, *Rk, *x, *r, *Sq, *Rq;
} fwd_scratch;

static int scratch_alloc(fwd_scratch *s, int64_t dv) {
    double *buf = (double *)calloc((size_t)(6 * dv), sizeof(double));
    if (!buf) return 0;
    s->Sk = buf; s->Rk = buf + dv; s->x = buf + 2 * dv; s->r = buf + 3 * dv;
    s->Sq = buf + 4 * dv; s->Rq = buf + 5 * dv;
    return 1;
}

/*
 * One token of the forward recurrence on states S, R ([dk][dv], transposed
 * storage).  Writes o (dv values) if o != NULL.  On return S = S_t, R = R_t.
 */
static void forward_token(int variant, int64_t dk, int64_t dv,
                          const double *q, const double *k, const double *v,
                          double aS, double b, double aR, double g, double c,
                          double *S, double *R, double *o, fwd_scratch *w) {
    int64_t i, j;
    const double eps = (variant & ORC_DECAYED) ? aS : 1.0;
    /* S_{t-1} k_t and the residual x_t = v_t - S_{t-1} k_t (DECAYED:
       v_t - aS_t S_{t-1} k_t), then r_t = phi(x_t). */
    for (j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (i = 0; i < dk; ++i) acc += S[i * dv + j] * k[i];
        w->Sk[j] = acc;
        w->x[j] = v[j] - eps * acc;
        w->r[j] = resid_value(variant, w->x[j], c);
    }
    /* R_t from R_{t-1}. */
    if (variant & ORC_RDN) {
        for (j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (i = 0; i < dk; ++i) acc += R[i * dv + j] * k[i];
            w->Rk[j] = acc;
        }
        for (i = 0; i < dk; ++i)
            for (j = 0; j < dv; ++j)
                R[i * dv + j] = aR * (R[i * dv + j] - g * k[i] * w->Rk[j]) + g * k[i] * w->r[j];
    } else {
        for (i = 0; i < dk; ++i)
            for (j = 0; j < dv; ++j)
                R[i * dv + j] = aR * R[i * dv + j] + g * k[i] * w->r[j];
    }
    /* o_t = aS S_{t-1} q_t + g R_t q_t (UNGATED: S_{t-1} q_t + R_t q_t). */
    if (o) {
        for (j = 0; j < dv; ++j) {
            double sq = 0.0, rq = 0.0;
            for (i = 0; i < dk; ++i) {
                sq += S[i * dv + j] * q[i];
                rq += R[i * dv + j] * q[i];
            }
            o[j] = (variant & ORC_UNGATED) ? sq + rq : aS * sq + g * rq;
        }
    }
    /* S_t from S_{t-1}. */
    if (variant & ORC_RDN) {
        for (i = 0; i < dk; ++i)
            for (j = 0; j < dv; ++j)
                S[i * dv + j] = aS * (S[i * dv + j] - b * k[i] * w->Sk[j]) + b * k[i] * v[j];
    } else {
        for (i = 0; i < dk; ++i)
            for (j = 0; j < dv; ++j)
                S[i * dv + j] = aS * S[i * dv + j] + b * k[i] * v[j];
    }
}

static int64_t clamp_i64(int64_t x, int64_t lo, int64_t hi) {
    return x < lo ? lo : (x > hi ? hi : x);
}

/*
 * Forward over all sequences and heads.
 * S0, R0 may be NULL (zero initial states); o, S_fin, R_fin may be NULL.
 * Returns 0 on success, nonzero on allocation failure.
 */
int orc_forward(int variant, int64_t nseq, const int64_t *cu, int64_t ntok,
                int64_t H, int64_t dk, int64_t dv,
                const double *q, const double *k, const double *v,
                const double *alpha_s, const double *beta,
                const double *alpha_r, const double *gamma, double clip,
                const double *S0, const double *R0,
                double *o, double *S_fin, double *R_fin) {
    int failed = 0;
    int64_t pair;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
    for (pair = 0; pair < nseq * H; ++pair) {
        int64_t n = pair / H, h = pair % H, t;
        int64_t t0 = clamp_i64(cu[n], 0, ntok), t1 = clamp_i64(cu[n + 1], t0, ntok);
        size_t ssz = (size_t)(dk * dv);
        double *S = (double *)calloc(ssz, sizeof(double));
        double *R = (double *)calloc(ssz, sizeof(double));
        fwd_scratch w;
        if (!S || !R || !scratch_alloc(&w, dv)) { failed |= 1; free(S); free(R); continue; }
        if (S0) memcpy(S, S0 + (n * H + h) * ssz, ssz * sizeof(double));
        if (R0) memcpy(R, R0 + (n * H + h) * ssz, ssz * sizeof(double));
        for (t = t0; t < t1; ++t) {
            int64_t th = t * H + h;
            forward_token(variant, dk, dv, q + th * dk, k + th * dk, v + th * dv,
                          alpha_s[th], beta[th], alpha_r[th], gamma[th], clip, S, R,
                          o ? o + th * dv : NULL, &w);
        }
        if (S_fin) memcpy(S_fin + (n * H + h) * ssz, S, ssz * sizeof(double));
        if (R_fin) memcpy(R_fin + (n * H + h) * ssz, R, ssz * sizeof(double));
        free(S); free(R); free(w.Sk);
    }
    return failed;
}

/*
 * Moves v so that no residual lies within `margin` of the clip kink (|x| = c).
 * Runs the forward recurrence; whenever | |x_t[j]| - c | < margin it shifts
 * v_t[j] (which leaves S_{t-1} untouched) to the nearest value at distance
 * >= margin from the kink, then rounds it away from the old value onto the
 * grid of the input dtype (round_bits = 16 keeps bf16 values, 0 keeps fp32
 * values, anything else keeps fp64), and continues with the moved v.
 * Returns the number of moved elements, or -1 on allocation failure.
 */
/* smallest fp32 value >= t */
static float f32_ceil(double t) {
    float f = (float)t;
    if ((double)f < t) f = nextafterf(f, INFINITY);
    return f;
}

/* smallest bf16 value >= t (bf16 = the upper 16 bits of an fp32) */
static double bf16_ceil(double t) {
    float f = f32_ceil(t), vz;
    uint32_t u, tz;
    memcpy(&u, &f, 4);
    tz = u & 0xFFFF0000u;            /* truncation: towards zero */
    memcpy(&vz, &tz, 4);
    if (f >= 0.0f && vz < f) {       /* positive and inexact: one step up */
        tz += 0x10000u;
        memcpy(&vz, &tz, 4);
    }
    return (double)vz;
}

/* the value on the input dtype's grid nearest to `target`, on the far side
 * of it as seen from `from` */
static double round_away(double target, double from, int round_bits) {
    if (round_bits == 16) return target > from ? bf16_ceil(target) : -bf16_ceil(-target);
    if (round_bits == 0) return target > from ? (double)f32_ceil(target) : -(double)f32_ceil(-target);
    return target;
}

int64_t orc_nudge_margin(int variant, int64_t nseq, const int64_t *cu, int64_t ntok,
                         int64_t H, int64_t dk, int64_t dv,
                         const double *q, const double *k, double *v,
                         const double *alpha_s, const double *beta,
                         const double *alpha_r, const double *gamma, double clip,
                         const double *S0, const double *R0, double margin, int round_bits) {
    int64_t moved = 0;
    int failed = 0;
    int64_t pair;
    if (clip < 0.0 || (variant & ORC_TANH)) return 0;   /* no kink */
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : moved) reduction(| : failed)
    for (pair = 0; pair < nseq * H; ++pair) {
        int64_t n = pair / H, h = pair % H, t, i, j;
        int64_t t0 = clamp_i64(cu[n], 0, ntok), t1 = clamp_i64(cu[n + 1], t0, ntok);
        size_t ssz = (size_t)(dk * dv);
        double *S = (double *)calloc(ssz, sizeof(double));
        double *R = (double *)calloc(ssz, sizeof(double));
        fwd_scratch w;
        if (!S || !R || !scratch_alloc(&w, dv)) { failed |= 1; free(S); free(R); continue; }
        if (S0) memcpy(S, S0 + (n * H + h) * ssz, ssz * sizeof(double));
        if (R0) memcpy(R, R0 + (n * H + h) * ssz, ssz * sizeof(double));
        for (t = t0; t < t1; ++t) {
            int64_t th = t * H + h;
            double *vt = v + th * dv;
            const double *kt = k + th * dk;
            for (j = 0; j < dv; ++j) {
                double p = 0.0;
                int tries;
                for (i = 0; i < dk; ++i) p += S[i * dv + j] * kt[i];
                if (variant & ORC_DECAYED) p *= alpha_s[th];
                for (tries = 0; tries < 8; ++tries) {
                    double x = vt[j] - p, ax = fabs(x), target_x, nv;
                    if (fabs(ax - clip) >= margin) break;
                    if (ax >= clip) target_x = (x >= 0 ? 1.0 : -1.0) * (clip + margin);
                    else if (clip - margin >= 0.0) target_x = (x >= 0 ? 1.0 : -1.0) * (clip - margin);
                    else target_x = (x >= 0 ? 1.0 : -1.0) * (clip + margin);
                    nv = round_away(p + target_x, vt[j], round_bits);
                    if (nv == vt[j]) break;
                    vt[j] = nv;
                    if (tries == 0) moved += 1;
                }
            }
            forward_token(variant, dk, dv, q + th * dk, kt, vt, alpha_s[th], beta[th],
                          alpha_r[th], gamma[th], clip, S, R, NULL, &w);
        }
        free(S); free(R); free(w.Sk);
    }
    return failed ? -1 : moved;
}

/*
 * Backward (vector-Jacobian product) of orc_forward for the scalar
 *   L = <do, o> + <dS_fin, S_T> + <dR_fin, R_T>.
 * dS_fin, dR_fin, S0, R0 may be NULL (zeros).  All gradient outputs are
 * overwritten.  dS0, dR0 may be NULL.  Gate gradients are with respect to the
 * gate values themselves.  Returns 0 on success.
 */
int orc_backward(int variant, int64_t nseq, const int64_t *cu, int64_t ntok,
                 int64_t H, int64_t dk, int64_t dv,
                 const double *q, const double *k, const double *v,
                 const double *alpha_s, const double *beta,
                 const double *alpha_r, const double *gamma, double clip,
                 const double *S0, const double *R0,
                 const double *dO, const double *dS_fin, const double *dR_fin,
                 double *dq, double *dk_out, double *dv_out,
                 double *dalpha_s, double *dbeta, double *dalpha_r, double *dgamma,
                 double *dS0, double *dR0) {
    int failed = 0;
    int64_t pair;
    memset(dq, 0, (size_t)(ntok * H * dk) * sizeof(double));
    memset(dk_out, 0, (size_t)(ntok * H * dk) * sizeof(double));
    memset(dv_out, 0, (size_t)(ntok * H * dv) * sizeof(double));
    memset(dalpha_s, 0, (size_t)(ntok * H) * sizeof(double));
    memset(dbeta, 0, (size_t)(ntok * H) * sizeof(double));
    memset(dalpha_r, 0, (size_t)(ntok * H) * sizeof(double));
    memset(dgamma, 0, (size_t)(ntok * H) * sizeof(double));
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
    for (pair = 0; pair < nseq * H; ++pair) {
        int64_t n = pair / H, h = pair % H;
        int64_t t0 = clamp_i64(cu[n], 0, ntok), t1 = clamp_i64(cu[n + 1], t0, ntok);
        int64_t L = t1 - t0, nck = (L + CKPT - 1) / CKPT, seg, t, i, j;
        size_t ssz = (size_t)(dk * dv);
        /* checkpoints: state before token t0 + s*CKPT, s = 0..nck-1 */
        double *ckS = (double *)malloc((size_t)(nck > 0 ? nck : 1) * ssz * sizeof(double));
        double *ckR = (double *)malloc((size_t)(nck > 0 ? nck : 1) * ssz * sizeof(double));
        /* per-token states before each token of one segment */
        double *segS = (double *)malloc((size_t)CKPT * ssz * sizeof(double));
        double *segR = (double *)malloc((size_t)CKPT * ssz * sizeof(double));
        double *S = (double *)calloc(ssz, sizeof(double));
        double *R = (double *)calloc(ssz, sizeof(double));
        double *dS = (double *)calloc(ssz, sizeof(double));
        double *dR = (double *)calloc(ssz, sizeof(double));
        double *dSp = (double *)calloc(ssz, sizeof(double));
        double *DR = (double *)calloc(ssz, sizeof(double));
        double *Rn = (double *)calloc(ssz, sizeof(double));
        double *vec = (double *)calloc((size_t)(10 * dv), sizeof(double));
        fwd_scratch w;
        if (!ckS || !ckR || !segS || !segR || !S || !R || !dS || !dR || !dSp || !DR || !Rn ||
            !vec || !scratch_alloc(&w, dv)) {
            failed |= 1;
            free(ckS); free(ckR); free(segS); free(segR); free(S); free(R); free(dS);
            free(dR); free(dSp); free(DR); free(Rn); free(vec);
            continue;
        }
        double *Sk = vec, *Rk = vec + dv, *x = vec + 2 * dv, *r = vec + 3 * dv, *z = vec + 4 * dv,
               *dr = vec + 5 * dv, *dx = vec + 6 * dv, *ww = vec + 7 * dv, *Sq = vec + 8 * dv,
               *Rq = vec + 9 * dv;
        if (S0) memcpy(S, S0 + (n * H + h) * ssz, ssz * sizeof(double));
        if (R0) memcpy(R, R0 + (n * H + h) * ssz, ssz * sizeof(double));
        for (t = t0; t < t1; ++t) {
            int64_t th = t * H + h;
            if ((t - t0) % CKPT == 0) {
                memcpy(ckS + ((t - t0) / CKPT) * ssz, S, ssz * sizeof(double));
                memcpy(ckR + ((t - t0) / CKPT) * ssz, R, ssz * sizeof(double));
            }
            forward_token(variant, dk, dv, q + th * dk, k + th * dk, v + th * dv, alpha_s[th],
                          beta[th], alpha_r[th], gamma[th], clip, S, R, NULL, &w);
        }
        if (dS_fin) memcpy(dS, dS_fin + (n * H + h) * ssz, ssz * sizeof(double));
        if (dR_fin) memcpy(dR, dR_fin + (n * H + h) * ssz, ssz * sizeof(double));
        for (seg = nck - 1; seg >= 0; --seg) {
            int64_t s0 = t0 + seg * CKPT, s1 = s0 + CKPT < t1 ? s0 + CKPT : t1;
            memcpy(S, ckS + seg * ssz, ssz * sizeof(double));
            memcpy(R, ckR + seg * ssz, ssz * sizeof(double));
            for (t = s0; t < s1; ++t) {
                int64_t th = t * H + h;
                memcpy(segS + (t - s0) * ssz, S, ssz * sizeof(double));
                memcpy(segR + (t - s0) * ssz, R, ssz * sizeof(double));
                forward_token(variant, dk, dv, q + th * dk, k + th * dk, v + th * dv,
                              alpha_s[th], beta[th], alpha_r[th], gamma[th], clip, S, R, NULL, &w);
            }
            for (t = s1 - 1; t >= s0; --t) {
                int64_t th = t * H + h;
                const double *Sp = segS + (t - s0) * ssz, *Rp = segR + (t - s0) * ssz;
                const double *qt = q + th * dk, *kt = k + th * dk, *vt = v + th * dv;
                const double *dot = dO + th * dv;
                double aS = alpha_s[th], b = beta[th], aR = alpha_r[th], g = gamma[th];
                double *dqt = dq + th * dk, *dkt = dk_out + th * dk, *dvt = dv_out + th * dv;
                double das = 0.0, dbb = 0.0, dar = 0.0, dg = 0.0;
                const double eps = (variant & ORC_DECAYED) ? aS : 1.0;
                const double wS = (variant & ORC_UNGATED) ? 1.0 : aS;   /* output weights */
                const double wR = (variant & ORC_UNGATED) ? 1.0 : g;
                /* recompute this token's forward quantities */
                for (j = 0; j < dv; ++j) {
                    double sk = 0.0, rk = 0.0, sq = 0.0;
                    for (i = 0; i < dk; ++i) {
                        sk += Sp[i * dv + j] * kt[i];
                        rk += Rp[i * dv + j] * kt[i];
                        sq += Sp[i * dv + j] * qt[i];
                    }
                    Sk[j] = sk; Rk[j] = rk; Sq[j] = sq;
                    x[j] = vt[j] - eps * sk;
                    r[j] = resid_value(variant, x[j], clip);
                }
                for (i = 0; i < dk; ++i)
                    for (j = 0; j < dv; ++j) {
                        if (variant & ORC_RDN)
                            Rn[i * dv + j] = aR * (Rp[i * dv + j] - g * kt[i] * Rk[j]) + g * kt[i] * r[j];
                        else
                            Rn[i * dv + j] = aR * Rp[i * dv + j] + g * kt[i] * r[j];
                    }
                for (j = 0; j < dv; ++j) {
                    double rq = 0.0;
                    for (i = 0; i < dk; ++i) rq += Rn[i * dv + j] * qt[i];
                    Rq[j] = rq;
                }
                /* output o_t = wS S_{t-1} q + wR R_t q (wS = aS, wR = g; UNGATED: 1, 1) */
                for (i = 0; i < dk; ++i) {
                    double a1 = 0.0, a2 = 0.0;
                    for (j = 0; j < dv; ++j) {
                        a1 += Sp[i * dv + j] * dot[j];
                        a2 += Rn[i * dv + j] * dot[j];
                    }
                    dqt[i] += wS * a1 + wR * a2;
                }
                if (!(variant & ORC_UNGATED)) {
                    for (j = 0; j < dv; ++j) {
                        das += dot[j] * Sq[j];
                        dg += dot[j] * Rq[j];
                    }
                }
                for (i = 0; i < dk; ++i)
                    for (j = 0; j < dv; ++j) {
                        DR[i * dv + j] = dR[i * dv + j] + wR * qt[i] * dot[j];
                        dSp[i * dv + j] = wS * qt[i] * dot[j];
                    }
                /* R update */
                for (j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (i = 0; i < dk; ++i) acc += DR[i * dv + j] * kt[i];
                    z[j] = acc;
                    dr[j] = g * acc;
                }
                if (variant & ORC_RDN) {
                    for (i = 0; i < dk; ++i) {
                        double rz = 0.0, drrk = 0.0, drr = 0.0;
                        for (j = 0; j < dv; ++j) {
                            dar += DR[i * dv + j] * (Rp[i * dv + j] - g * kt[i] * Rk[j]);
                            rz += Rp[i * dv + j] * z[j];
                            drrk += DR[i * dv + j] * Rk[j];
                            drr += DR[i * dv + j] * r[j];
                        }
                        dkt[i] += -aR * g * (rz + drrk) + g * drr;
                    }
                    for (j = 0; j < dv; ++j) dg += z[j] * (r[j] - aR * Rk[j]);
                    for (i = 0; i < dk; ++i)
                        for (j = 0; j < dv; ++j)
                            dR[i * dv + j] = aR * (DR[i * dv + j] - g * kt[i] * z[j]);
                } else {
                    for (i = 0; i < dk; ++i) {
                        double drr = 0.0;
                        for (j = 0; j < dv; ++j) {
                            dar += DR[i * dv + j] * Rp[i * dv + j];
                            drr += DR[i * dv + j] * r[j];
                        }
                        dkt[i] += g * drr;
                    }
                    for (j = 0; j < dv; ++j) dg += z[j] * r[j];
                    for (i = 0; i < dk; ++i)
                        for (j = 0; j < dv; ++j) dR[i * dv + j] = aR * DR[i * dv + j];
                }
                /* residual function, then x = v - eps S_{t-1} k */
                for (j = 0; j < dv; ++j) {
                    dx[j] = resid_slope(variant, x[j], clip) * dr[j];
                    dvt[j] += dx[j];
                    if (variant & ORC_DECAYED) das -= dx[j] * Sk[j];
                }
                for (i = 0; i < dk; ++i) {
                    double acc = 0.0;
                    for (j = 0; j < dv; ++j) {
                        dSp[i * dv + j] -= eps * kt[i] * dx[j];
                        acc += Sp[i * dv + j] * dx[j];
                    }
                    dkt[i] -= eps * acc;
                }
                /* S update */
                for (j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (i = 0; i < dk; ++i) acc += dS[i * dv + j] * kt[i];
                    ww[j] = acc;
                }
                if (variant & ORC_RDN) {
                    for (i = 0; i < dk; ++i) {
                        double sw = 0.0, dssk = 0.0, dsv = 0.0;
                        for (j = 0; j < dv; ++j) {
                            das += dS[i * dv + j] * (Sp[i * dv + j] - b * kt[i] * Sk[j]);
                            sw += Sp[i * dv + j] * ww[j];
                            dssk += dS[i * dv + j] * Sk[j];
                            dsv += dS[i * dv + j] * vt[j];
                            dSp[i * dv + j] += aS * (dS[i * dv + j] - b * kt[i] * ww[j]);
                        }
                        dkt[i] += -aS * b * (sw + dssk) + b * dsv;
                    }
                    for (j = 0; j < dv; ++j) {
                        dbb += ww[j] * (vt[j] - aS * Sk[j]);
                        dvt[j] += b * ww[j];
                    }
                } else {
                    for (i = 0; i < dk; ++i) {
                        double dsv = 0.0;
                        for (j = 0; j < dv; ++j) {
                            das += dS[i * dv + j] * Sp[i * dv + j];
                            dsv += dS[i * dv + j] * vt[j];
                            dSp[i * dv + j] += aS * dS[i * dv + j];
                        }
                        dkt[i] += b * dsv;
                    }
                    for (j = 0; j < dv; ++j) {
                        dbb += ww[j] * vt[j];
                        dvt[j] += b * ww[j];
                    }
                }
                memcpy(dS, dSp, ssz * sizeof(double));
                dalpha_s[th] = das;
                dbeta[th] = dbb;
                dalpha_r[th] = dar;
                dgamma[th] = dg;
            }
        }
        if (dS0) memcpy(dS0 + (n * H + h) * ssz, dS, ssz * sizeof(double));
        if (dR0) memcpy(dR0 + (n * H + h) * ssz, dR, ssz * sizeof(double));
        free(ckS); free(ckR); free(segS); free(segR); free(S); free(R); free(dS); free(dR);
        free(dSp); free(DR); free(Rn); free(vec); free(w.Sk);
    }
    return failed;
}

int orc_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
