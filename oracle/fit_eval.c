/*
 * Candidate scoring for the oracle's continuous groupwise fitter.
 *
 * TEST INFRASTRUCTURE ONLY: compiled with gcc into oracle/_fit_eval.so and
 * called from oracle/fit.py.  The product library never links it.
 *
 * For one weight group and one shape candidate (a, b) it minimises the
 * original-domain squared error of Sec. 4.1 (eq. offline-objective) over the
 * scale s and the codes: s is both the endpoint and the clipping threshold,
 * every magnitude is assigned to its nearest continuous level s*q(i/M)
 * (midpoint boundaries, ties to the smaller magnitude), and the scale is the
 * least-squares optimum for the current assignment.  Everything is float64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MAXLEV 128

static void make_levels(int m, double a, double b, double *z) {
    double c = 1.0 - a - b;
    for (int i = 0; i <= m; ++i) {
        double t = (double)i / (double)m;
        z[i] = t * (a + t * (b + t * c));
    }
}

/* nearest level index for magnitude u with scale s: the number of midpoint
 * boundaries h_i = s (z_i + z_{i+1}) / 2 that lie strictly below u. */
static int assign(double u, double s, const double *mid, int m) {
    int lo = 0, hi = m; /* answer in [0, m] */
    while (lo < hi) {
        int mid_i = (lo + hi) >> 1;
        if (u > s * mid[mid_i]) lo = mid_i + 1; else hi = mid_i;
    }
    return lo;
}

/* Number of sorted magnitudes su[lo..g) that are <= h, plus lo. */
static int upper_pos(const double *su, int lo, int g, double h) {
    int hi = g;
    while (lo < hi) {
        int mid_i = (lo + hi) >> 1;
        if (su[mid_i] <= h) lo = mid_i + 1; else hi = mid_i;
    }
    return lo;
}

/* Score one candidate on one group.  su holds the magnitudes sorted
 * ascending and p1/p2 their prefix sums of u and u^2, so that the nearest-
 * level cells (boundaries h_i = s (z_i + z_{i+1}) / 2, a magnitude equal to a
 * boundary going to the smaller level) are index ranges of su.  Returns the
 * SSE and the scale. */
static double score(const double *su, const double *p1, const double *p2, int g,
                    int m, double a, double b, const double *clips, int nclips,
                    int iters, double umax, double *s_out) {
    double z[MAXLEV + 1], mid[MAXLEV];
    int pos[MAXLEV + 2];
    make_levels(m, a, b, z);
    for (int i = 0; i < m; ++i) mid[i] = 0.5 * (z[i] + z[i + 1]);
    double best = INFINITY, best_s = 0.0;
    for (int ci = 0; ci < nclips; ++ci) {
        double s = clips[ci] * umax;
        for (int it = 0; it <= iters; ++it) {
            /* cell i holds sorted indices [pos[i], pos[i+1]) */
            pos[0] = 0;
            for (int i = 0; i < m; ++i) pos[i + 1] = upper_pos(su, pos[i], g, s * mid[i]);
            pos[m + 1] = g;
            double num = 0.0, den = 0.0, sse = 0.0;
            for (int i = 0; i <= m; ++i) {
                int n0 = pos[i], n1 = pos[i + 1];
                if (n1 <= n0) continue;
                double s1 = p1[n1] - p1[n0], s2 = p2[n1] - p2[n0], cnt = (double)(n1 - n0);
                num += z[i] * s1;
                den += z[i] * z[i] * cnt;
                sse += s2 - 2.0 * s * z[i] * s1 + s * s * z[i] * z[i] * cnt;
            }
            if (it == iters) {
                if (sse < best) { best = sse; best_s = s; }
            } else if (den > 0.0) {
                s = num / den;
            }
        }
    }
    *s_out = best_s;
    return best;
}

static int cmp_double(const void *x, const void *y) {
    double a = *(const double *)x, b = *(const double *)y;
    return (a > b) - (a < b);
}

/*
 * Evaluate per-group candidate lists.
 *   w        [ngroups * g] float32 weights
 *   cand_a/b [ngroups * ncand] (or [ncand] when shared != 0) float64 shapes
 *   valid    same shape as cand_a, nonzero where the candidate is admissible
 * For every group the lowest-SSE candidate wins; ties keep the earlier one.
 * Outputs best index (-1 if none valid), its SSE and its scale.
 */
int cq_oracle_eval_candidates(const float *w, int64_t ngroups, int g, int bits,
                              const double *cand_a, const double *cand_b,
                              const uint8_t *valid, int ncand, int shared,
                              const double *clips, int nclips, int iters,
                              int32_t *best_idx, double *best_sse, double *best_s) {
    if (bits < 2 || bits > 8 || g <= 0 || g > 4096) return 1;
    int m = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t gi = 0; gi < ngroups; ++gi) {
        double su[4096], p1[4097], p2[4097];
        double umax = 0.0;
        for (int j = 0; j < g; ++j) {
            su[j] = fabs((double)w[gi * g + j]);
            if (su[j] > umax) umax = su[j];
        }
        qsort(su, (size_t)g, sizeof(double), cmp_double);
        p1[0] = 0.0; p2[0] = 0.0;
        for (int j = 0; j < g; ++j) { p1[j + 1] = p1[j] + su[j]; p2[j + 1] = p2[j] + su[j] * su[j]; }
        int32_t bi = -1;
        double bsse = INFINITY, bs = 0.0;
        for (int c = 0; c < ncand; ++c) {
            int64_t off = shared ? c : gi * (int64_t)ncand + c;
            if (!valid[off]) continue;
            double s;
            double sse = score(su, p1, p2, g, m, cand_a[off], cand_b[off], clips, nclips,
                               iters, umax, &s);
            if (sse < bsse) { bsse = sse; bs = s; bi = c; }
        }
        best_idx[gi] = bi;
        best_sse[gi] = bsse;
        best_s[gi] = bs;
    }
    return 0;
}

/*
 * Final code assignment for the serialized representation: nearest level of
 * |w| under the stored float32 scale and float16 shapes, signed by w (w = 0
 * gives code 0).  Also returns the group SSE of the serialized codes.
 */
int cq_oracle_assign_serialized(const float *w, int64_t ngroups, int g, int bits,
                                const float *s, const double *a, const double *b,
                                int8_t *codes, double *sse_out) {
    if (bits < 2 || bits > 8 || g <= 0) return 1;
    int m = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(static)
    for (int64_t gi = 0; gi < ngroups; ++gi) {
        double z[MAXLEV + 1], mid[MAXLEV];
        make_levels(m, a[gi], b[gi], z);
        for (int i = 0; i < m; ++i) mid[i] = 0.5 * (z[i] + z[i + 1]);
        double sc = (double)s[gi], sse = 0.0;
        for (int j = 0; j < g; ++j) {
            double wv = (double)w[gi * g + j];
            double u = fabs(wv);
            int i = (sc > 0.0) ? assign(u, sc, mid, m) : 0;
            int k = (wv > 0.0) ? i : (wv < 0.0 ? -i : 0);
            codes[gi * g + j] = (int8_t)k;
            double e = u - sc * z[i];
            sse += e * e;
        }
        sse_out[gi] = sse;
    }
    return 0;
}

/* ------------------------------------------------------------------ joint
 * Carrier-aware joint objective (Sec. 4.3, eq. carrier-aware-objective):
 * L_C + L_A8 with the continuous levels z_i = q(i/M) and the carrier levels
 * zt_i = RNE(127 z_i) / 127 (eq. carrier-grid), the carrier rounded from the
 * exact rational value of the FP16 shapes.  Codes take the argmin of
 * (u - s z_i)^2 + (u - s zt_i)^2 over i (eq. carrier-aware-assignment, ties
 * to the smaller magnitude), the scale the closed form
 * s = sum u (z + zt) / sum (z^2 + zt^2) (eq. carrier-aware-scale).
 */

/* RNE(127 q(i/m)) from FP16 shape values a, b: with A = 2^24 a and
 * Bq = 2^24 b (integers, FP16 values being multiples of 2^-24) and
 * C = 2^24 - A - Bq, 127 q(i/m) = 127 (A i m^2 + Bq i^2 m + C i^3) / (2^24 m^3),
 * an exact rational with an int64 numerator for m <= 127. */
static int carrier_exact(int i, int m, double a, double b) {
    const int64_t A = (int64_t)llround(a * 16777216.0), Bq = (int64_t)llround(b * 16777216.0);
    const int64_t C = ((int64_t)1 << 24) - A - Bq;
    const int64_t ii = i, mm = m;
    const int64_t num = 127 * (A * ii * mm * mm + Bq * ii * ii * mm + C * ii * ii * ii);
    const int64_t den = ((int64_t)1 << 24) * mm * mm * mm;
    /* nearest integer to num / den, ties to even (num >= 0 for admissible shapes) */
    int64_t qt = num / den, r = num - qt * den;
    if (r < 0) { qt -= 1; r += den; }
    if (2 * r > den || (2 * r == den && (qt & 1))) qt += 1;
    return (int)qt;
}

int cq_oracle_carriers(int bits, double a, double b, int32_t *out) {
    if (bits < 2 || bits > 8) return 1;
    int m = (1 << (bits - 1)) - 1;
    for (int i = 0; i <= m; ++i) out[i] = carrier_exact(i, m, a, b);
    return 0;
}

static void make_joint_levels(int m, double a, double b, double *z, double *zt) {
    make_levels(m, a, b, z);
    for (int i = 0; i <= m; ++i) zt[i] = (double)carrier_exact(i, m, a, b) / 127.0;
}

static int assign_joint(double u, double s, const double *z, const double *zt, int m) {
    int best = 0;
    double bc = INFINITY;
    for (int i = 0; i <= m; ++i) {
        double e1 = u - s * z[i], e2 = u - s * zt[i];
        double c = e1 * e1 + e2 * e2;
        if (c < bc) { bc = c; best = i; }
    }
    return best;
}

static double score_joint(const double *u, int g, int m, double a, double b, const double *clips, int nclips,
                          int iters, double umax, double *s_out) {
    double z[MAXLEV + 1], zt[MAXLEV + 1];
    make_joint_levels(m, a, b, z, zt);
    double best = INFINITY, best_s = 0.0;
    for (int ci = 0; ci < nclips; ++ci) {
        double s = clips[ci] * umax;
        for (int it = 0; it <= iters; ++it) {
            double num = 0.0, den = 0.0, loss = 0.0;
            for (int j = 0; j < g; ++j) {
                int i = assign_joint(u[j], s, z, zt, m);
                num += u[j] * (z[i] + zt[i]);
                den += z[i] * z[i] + zt[i] * zt[i];
                double e1 = u[j] - s * z[i], e2 = u[j] - s * zt[i];
                loss += e1 * e1 + e2 * e2;
            }
            if (it == iters) {
                if (loss < best) { best = loss; best_s = s; }
            } else if (den > 0.0) {
                s = num / den;
            }
        }
    }
    *s_out = best_s;
    return best;
}

/* As cq_oracle_eval_candidates, scoring L_C + L_A8. */
int cq_oracle_eval_candidates_joint(const float *w, int64_t ngroups, int g, int bits,
                                    const double *cand_a, const double *cand_b,
                                    const uint8_t *valid, int ncand, int shared,
                                    const double *clips, int nclips, int iters,
                                    int32_t *best_idx, double *best_loss, double *best_s) {
    if (bits < 2 || bits > 8 || g <= 0 || g > 4096) return 1;
    int m = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t gi = 0; gi < ngroups; ++gi) {
        double u[4096];
        double umax = 0.0;
        for (int j = 0; j < g; ++j) {
            u[j] = fabs((double)w[gi * g + j]);
            if (u[j] > umax) umax = u[j];
        }
        int32_t bi = -1;
        double bl = INFINITY, bs = 0.0;
        for (int c = 0; c < ncand; ++c) {
            int64_t off = shared ? c : gi * (int64_t)ncand + c;
            if (!valid[off]) continue;
            double s;
            double l = score_joint(u, g, m, cand_a[off], cand_b[off], clips, nclips, iters, umax, &s);
            if (l < bl) { bl = l; bs = s; bi = c; }
        }
        best_idx[gi] = bi;
        best_loss[gi] = bl;
        best_s[gi] = bs;
    }
    return 0;
}

/* Final joint assignment under the stored FP32 scale and FP16 shapes, with the
 * carriers given per group (carriers[gi * (m + 1) + i], from the caller's
 * exact carrier table).  Returns the signed codes and, per group, L_C and L_A8. */
int cq_oracle_assign_serialized_joint(const float *w, int64_t ngroups, int g, int bits,
                                      const float *s, const double *a, const double *b,
                                      const int32_t *carriers, int8_t *codes, double *lc_out, double *la8_out) {
    if (bits < 2 || bits > 8 || g <= 0) return 1;
    int m = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(static)
    for (int64_t gi = 0; gi < ngroups; ++gi) {
        double z[MAXLEV + 1], zt[MAXLEV + 1];
        make_levels(m, a[gi], b[gi], z);
        for (int i = 0; i <= m; ++i) zt[i] = (double)carriers[gi * (int64_t)(m + 1) + i] / 127.0;
        double sc = (double)s[gi], lc = 0.0, la = 0.0;
        for (int j = 0; j < g; ++j) {
            double wv = (double)w[gi * g + j];
            double u = fabs(wv);
            int i = (sc > 0.0) ? assign_joint(u, sc, z, zt, m) : 0;
            int k = (wv > 0.0) ? i : (wv < 0.0 ? -i : 0);
            codes[gi * g + j] = (int8_t)k;
            double e1 = u - sc * z[i], e2 = u - sc * zt[i];
            lc += e1 * e1;
            la += e2 * e2;
        }
        lc_out[gi] = lc;
        la8_out[gi] = la;
    }
    return 0;
}
