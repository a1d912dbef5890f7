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
