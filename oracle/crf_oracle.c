/*
 * crf_oracle.c -- float64 CPU oracle for the span-based tree CRF.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * GPU path is checked against.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load it; the product library never links it
 * and shares no code, header or table with it.
 *
 * Method: Zhang, Zhou & Li, "Fast and Accurate Neural CRF Constituency
 * Parsing" (IJCAI 2020).
 *   - tree score s(x,y) = sum of the scores of the spans of y       (Sec. 2.1, Eq. tree-score)
 *   - p(y|x) = exp(s(x,y)) / Z(x), Z summing over all legal trees    (Sec. 2.1, Eq. tree-prob)
 *   - Z by the inside recursion over span widths                     (Sec. 3.1, Algorithm 1)
 *   - span marginals = d log Z / d s(i,j)                            (Sec. 3.2, Eq. partial-derivative)
 *   - 1-best tree by CKY: the same recursion with max for sum        (Sec. 3.3; Sec. 2.1, Eq. tree-argmax)
 *   - one-stage labelled score: sum of s(i,j,l) over labelled spans  (Sec. 4.2, Eq. tree-label-score)
 *
 * Conventions.  Fence posts: a sentence of n words has boundaries 0..n and the
 * span (i,j), 0 <= i < j <= n, covers words i..j-1 (the paper's inclusive
 * (i, j-1)).  Width-1 spans are scored, since every CNF tree contains each
 * single-word constituent (Sec. 2.1: every CNF tree has 2n-1 constituents;
 * Fig. 1b).  One sentence's scores sit in a row-major ld x ld block with
 * s(i,j) at [i*ld + j]; no other cell is ever read (padding may hold NaN).
 * All arithmetic is IEEE float64; log-sum-exp is evaluated with a max shift.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define IDX(i, j, stride) ((size_t)(i) * (size_t)(stride) + (size_t)(j))

/* log(sum_k exp(x[k])) for m >= 1 finite-or--inf terms, max-shifted. */
static double log_sum_exp(const double *x, int m)
{
    double mx = -INFINITY;
    for (int k = 0; k < m; ++k)
        if (x[k] > mx) mx = x[k];
    if (mx == -INFINITY) return -INFINITY;
    double acc = 0.0;
    for (int k = 0; k < m; ++k) acc += exp(x[k] - mx);
    return mx + log(acc);
}

/* ------------------------------------------------------------------------ */
/* Inside (Sec. 3.1, Algorithm 1, read with fence posts and scored width-1
 * spans):  alpha(i,i+1) = s(i,i+1);  for w = 2..n,
 *   alpha(i,j) = s(i,j) + log sum_{i<k<j} exp(alpha(i,k) + alpha(k,j)),
 * and log Z = alpha(0,n).  alpha has stride n+1.  Returns log Z.           */
static double inside(int n, int ld, const double *s, double *alpha, double *tmp)
{
    const int st = n + 1;
    for (int i = 0; i < n; ++i) alpha[IDX(i, i + 1, st)] = s[IDX(i, i + 1, ld)];
    for (int w = 2; w <= n; ++w) {
        for (int i = 0; i + w <= n; ++i) {
            const int j = i + w;
            int m = 0;
            for (int k = i + 1; k < j; ++k)
                tmp[m++] = alpha[IDX(i, k, st)] + alpha[IDX(k, j, st)];
            alpha[IDX(i, j, st)] = s[IDX(i, j, ld)] + log_sum_exp(tmp, m);
        }
    }
    return alpha[IDX(0, n, st)];
}

/* ------------------------------------------------------------------------ */
/* Marginals, derivation 1: the classical outside pass in log space.  The
 * outside score O(i,j) sums, over all trees containing (i,j), everything
 * outside the subtree of (i,j).  O(0,n) = 0; a span (i,k) is the left child
 * of a parent (i,j), j > k, whose other child is (k,j), or the right child of
 * a parent (m,k), m < i, whose other child is (m,i):
 *   O(i,k) = log [ sum_{j>k} exp(O(i,j) + s(i,j) + alpha(k,j))
 *                + sum_{m<i} exp(O(m,k) + s(m,k) + alpha(m,i)) ].
 * Then p((i,j)|x) = exp(alpha(i,j) + O(i,j) - log Z)   (Eq. partial-derivative). */
static void outside_marginals(int n, int ld, const double *s, const double *alpha,
                              double logZ, double g, double *O, double *tmp,
                              double *mu)
{
    const int st = n + 1;
    for (size_t c = 0; c < (size_t)st * st; ++c) O[c] = -INFINITY;
    O[IDX(0, n, st)] = 0.0;
    for (int w = n - 1; w >= 1; --w) {
        for (int i = 0; i + w <= n; ++i) {
            const int k = i + w;
            int m = 0;
            for (int j = k + 1; j <= n; ++j)
                tmp[m++] = O[IDX(i, j, st)] + s[IDX(i, j, ld)] + alpha[IDX(k, j, st)];
            for (int a = 0; a < i; ++a)
                tmp[m++] = O[IDX(a, k, st)] + s[IDX(a, k, ld)] + alpha[IDX(a, i, st)];
            O[IDX(i, k, st)] = log_sum_exp(tmp, m);
        }
    }
    for (int i = 0; i < n; ++i)
        for (int j = i + 1; j <= n; ++j)
            mu[IDX(i, j, ld)] = g * exp(alpha[IDX(i, j, st)] + O[IDX(i, j, st)] - logZ);
}

/* ------------------------------------------------------------------------ */
/* Marginals, derivation 2: reverse-mode differentiation of the inside
 * recursion, which is how the paper obtains them (Sec. 3.2).  With
 * gbar(x) = d(g * log Z)/dx: gbar(alpha(0,n)) = g; processing widths from n
 * down to 2, each span's adjoint is complete when it is reached, equals
 * d(g log Z)/d s(i,j) because alpha(i,j) = s(i,j) + LSE(...), and flows to
 * both children of each split k with the softmax weight of that split:
 *   p_k = exp(alpha(i,k) + alpha(k,j) - LSE_k'(alpha(i,k') + alpha(k',j))).  */
static void adjoint_marginals(int n, int ld, const double *alpha, double g,
                              double *gbar, double *tmp, double *mu)
{
    const int st = n + 1;
    for (size_t c = 0; c < (size_t)st * st; ++c) gbar[c] = 0.0;
    gbar[IDX(0, n, st)] = g;
    for (int w = n; w >= 2; --w) {
        for (int i = 0; i + w <= n; ++i) {
            const int j = i + w;
            const double a = gbar[IDX(i, j, st)];
            mu[IDX(i, j, ld)] = a;
            int m = 0;
            for (int k = i + 1; k < j; ++k)
                tmp[m++] = alpha[IDX(i, k, st)] + alpha[IDX(k, j, st)];
            const double lse = log_sum_exp(tmp, m);
            for (int k = i + 1; k < j; ++k) {
                const double p = exp(tmp[k - i - 1] - lse);
                gbar[IDX(i, k, st)] += a * p;
                gbar[IDX(k, j, st)] += a * p;
            }
        }
    }
    for (int i = 0; i < n; ++i) mu[IDX(i, i + 1, ld)] = gbar[IDX(i, i + 1, st)];
}

/* ------------------------------------------------------------------------ */
/* CKY (Sec. 3.3: the inside recursion with max in place of log-sum-exp;
 * Eq. tree-argmax).  beta(i,i+1) = s(i,i+1);
 *   beta(i,j) = (max_{i<k<j} (beta(i,k) + beta(k,j))) + s(i,j),
 * evaluated in exactly that association order.  The split kept is the lowest
 * k attaining the maximum (strict '>' while scanning k upwards).  The tree is
 * written in preorder (parent, then left subtree, then right subtree), which
 * is the order of the spans sorted by i ascending, then j descending:
 * exactly 2n-1 rows of (i,j).  Returns beta(0,n), the best tree's score.    */
static double cky(int n, int ld, const double *s, double *beta, int32_t *bp,
                  int32_t *stack, int32_t *spans)
{
    const int st = n + 1;
    for (int i = 0; i < n; ++i) beta[IDX(i, i + 1, st)] = s[IDX(i, i + 1, ld)];
    for (int w = 2; w <= n; ++w) {
        for (int i = 0; i + w <= n; ++i) {
            const int j = i + w;
            double best = -INFINITY;
            int bk = -1;
            for (int k = i + 1; k < j; ++k) {
                const double v = beta[IDX(i, k, st)] + beta[IDX(k, j, st)];
                if (bk < 0 || v > best) { best = v; bk = k; }
            }
            beta[IDX(i, j, st)] = best + s[IDX(i, j, ld)];
            bp[IDX(i, j, st)] = bk;
        }
    }
    int top = 0, row = 0;
    stack[top++] = 0; stack[top++] = n;
    while (top > 0) {
        const int j = stack[--top];
        const int i = stack[--top];
        spans[2 * row] = i; spans[2 * row + 1] = j; ++row;
        if (j - i > 1) {
            const int k = bp[IDX(i, j, st)];
            stack[top++] = k; stack[top++] = j;   /* right child, popped second */
            stack[top++] = i; stack[top++] = k;   /* left child, popped first   */
        }
    }
    return beta[IDX(0, n, st)];
}

/* ------------------------------------------------------------------------ */
/* Second stage of the two-stage parser, labelling (Sec. 2.1, Eq. label-argmax):
 * every span of a given tree independently takes argmax_l s(i,j,l).  Among
 * equal maxima the lowest label index is kept.  s4 points at one sentence's
 * [ld][ld][L] block.                                                        */
static int32_t best_label(const float *s4, int ld, int L, int i, int j)
{
    const float *v = s4 + IDX(i, j, ld) * (size_t)L;
    int32_t bl = 0;
    for (int l = 1; l < L; ++l)
        if (v[l] > v[bl]) bl = l;
    return bl;
}

/* Whether (i,j) is a span of an n-word sentence. */
static int valid_span(int n, int i, int j) { return 0 <= i && i < j && j <= n; }

/* ------------------------------------------------------------------------ */
/* Batch drivers.  Sentences are independent (Algorithm 1 parallelises over
 * the batch), so worker threads take whole sentences from a shared counter. */

enum { JOB_LOGZ = 0, JOB_MARG_ADJ = 1, JOB_MARG_OUT = 2, JOB_CKY = 3, JOB_LABEL = 4, JOB_LOSS = 5,
       JOB_LCKY = 6, JOB_LSPANS = 7 };

typedef struct {
    int job, B, ld, L;
    const int32_t *len;
    const float *s;          /* [B][ld][ld] or [B][ld][ld][L] */
    const double *g;         /* [B] upstream gradient, NULL = 1 */
    double *logZ;            /* [B] (or best score for CKY, loss for JOB_LOSS), may be NULL */
    double *mu;              /* [B][ld][ld] or [B][ld][ld][L], may be NULL */
    int32_t *spans;          /* [B][2(ld-1)-1][2] (input for JOB_LOSS and JOB_LSPANS) */
    int32_t *labels;         /* [B][2(ld-1)-1] (JOB_LCKY, JOB_LSPANS) */
    volatile int next;
    volatile int status;
} job_t;

static void run_one(job_t *J, int b, double *buf)
{
    const int n = J->len[b], ld = J->ld, st = n + 1;
    const size_t blk = (size_t)ld * ld;
    double *sd = buf;                          /* ld*ld: scores as float64   */
    double *c1 = sd + blk;                     /* st*st: alpha / beta        */
    double *c2 = c1 + (size_t)st * st;         /* st*st: outside / adjoint   */
    double *tmp = c2 + (size_t)st * st;        /* 2*st scratch terms         */
    const double g = J->g ? J->g[b] : 1.0;

    const int R = 2 * (ld - 1) - 1;   /* rows of a span list */

    if (J->job == JOB_LSPANS) {
        /* Labelling stage on a given tree: every listed row that is a span of
         * this sentence gets its best label; every other row gets -1.       */
        const float *s4 = J->s + (size_t)b * blk * J->L;
        const int32_t *sp = J->spans + (size_t)b * R * 2;
        int32_t *lab = J->labels + (size_t)b * R;
        for (int r = 0; r < R; ++r)
            lab[r] = valid_span(n, sp[2 * r], sp[2 * r + 1]) ? best_label(s4, ld, J->L, sp[2 * r], sp[2 * r + 1]) : -1;
        return;
    }

    if (J->job == JOB_LCKY) {
        /* One-stage labelled decoding (Sec. 4.2, Eq. tree-label-score; the
         * time-complexity paragraph of Sec. 2.1: CKY picks the best label of
         * every span).  A labelled tree scores the sum of s(i,j,l) over its
         * labelled spans, and each span's label is free, so the best labelled
         * tree is the CKY tree over s'(i,j) = max_l s(i,j,l) with each of its
         * spans labelled argmax_l s(i,j,l) (lowest label on ties).  s' is a
         * float32 value (an exact max), decoded by the float64 CKY above.   */
        const int L = J->L;
        const float *s4 = J->s + (size_t)b * blk * L;
        for (int i = 0; i < n; ++i)
            for (int j = i + 1; j <= n; ++j)
                sd[IDX(i, j, ld)] = (double)s4[IDX(i, j, ld) * L + best_label(s4, ld, L, i, j)];
        int32_t *bp = (int32_t *)c2;
        int32_t *stack = (int32_t *)tmp;
        int32_t *sp = J->spans + (size_t)b * R * 2;
        int32_t *lab = J->labels + (size_t)b * R;
        for (int r = 0; r < R * 2; ++r) sp[r] = -1;
        const double best = cky(n, ld, sd, c1, bp, stack, sp);
        for (int r = 0; r < R; ++r) lab[r] = r < 2 * n - 1 ? best_label(s4, ld, L, sp[2 * r], sp[2 * r + 1]) : -1;
        if (J->logZ) J->logZ[b] = best;
        return;
    }

    if (J->job == JOB_LABEL) {
        /* One-stage labelled CRF (Sec. 4.2, Eq. tree-label-score): a tree's
         * labelled score sums s(i,j,l) over its labelled spans, so
         *   Z = sum_y prod_{(i,j) in y} sum_l exp(s(i,j,l)),
         * i.e. the unlabelled inside on s'(i,j) = log sum_l exp(s(i,j,l)),
         * and p((i,j,l)|x) = p((i,j)|x) * exp(s(i,j,l) - s'(i,j)).          */
        const int L = J->L;
        const float *s4 = J->s + (size_t)b * blk * L;
        for (int i = 0; i < n; ++i)
            for (int j = i + 1; j <= n; ++j) {
                double mx = -INFINITY;
                for (int l = 0; l < L; ++l) {
                    double v = s4[IDX(i, j, ld) * L + l];
                    if (v > mx) mx = v;
                }
                double acc = 0.0;
                for (int l = 0; l < L; ++l) acc += exp((double)s4[IDX(i, j, ld) * L + l] - mx);
                sd[IDX(i, j, ld)] = mx + log(acc);
            }
        const double lz = inside(n, ld, sd, c1, tmp);
        if (J->logZ) J->logZ[b] = lz;
        if (J->mu) {
            double *mu2 = (double *)malloc(blk * sizeof(double));
            if (!mu2) { J->status = 2; return; }
            adjoint_marginals(n, ld, c1, g, c2, tmp, mu2);
            double *m4 = J->mu + (size_t)b * blk * L;
            for (int i = 0; i < n; ++i)
                for (int j = i + 1; j <= n; ++j)
                    for (int l = 0; l < L; ++l)
                        m4[IDX(i, j, ld) * L + l] =
                            mu2[IDX(i, j, ld)] *
                            exp((double)s4[IDX(i, j, ld) * L + l] - sd[IDX(i, j, ld)]);
            free(mu2);
        }
        return;
    }

    const float *sb = J->s + (size_t)b * blk;
    for (int i = 0; i < n; ++i)
        for (int j = i + 1; j <= n; ++j) sd[IDX(i, j, ld)] = (double)sb[IDX(i, j, ld)];

    if (J->job == JOB_CKY) {
        int32_t *bp = (int32_t *)c2;             /* st*st int32 fits in st*st doubles */
        int32_t *stack = (int32_t *)tmp;         /* depth <= n+1 pairs; tmp has 2*st doubles */
        const int rows = 2 * (ld - 1) - 1;
        int32_t *sp = J->spans + (size_t)b * rows * 2;
        for (int r = 0; r < rows * 2; ++r) sp[r] = -1;
        const double best = cky(n, ld, sd, c1, bp, stack, sp);
        if (J->logZ) J->logZ[b] = best;
        return;
    }

    const double lz = inside(n, ld, sd, c1, tmp);
    if (J->job == JOB_LOSS) {
        /* Gold-tree CRF loss (Sec. 2.3, Eq. bracket-loss):
         *   L = -s(x,y) + log Z(x),  s(x,y) = sum of the scores of y's spans
         * (Eq. tree-score), and its gradient, the marginals minus the gold
         * indicator: dL/ds(i,j) = p((i,j)|x) - 1[(i,j) in y] (Sec. 3.2),
         * the gradient times the upstream gradient g.  y is the set of the first
         * 2n-1 rows of the span list; every one must be a span of this
         * sentence (else the job fails); a repeated row adds its score again
         * but the indicator of a set.                                        */
        const int32_t *gy = J->spans + (size_t)b * R * 2;
        double *mu = J->mu + (size_t)b * blk;
        adjoint_marginals(n, ld, c1, g, c2, tmp, mu);
        char *hit = (char *)c2;               /* c2 is free again: st*st flags */
        memset(hit, 0, (size_t)st * st);
        double gold = 0.0;
        for (int r = 0; r < 2 * n - 1; ++r) {
            const int i = gy[2 * r], j = gy[2 * r + 1];
            if (!valid_span(n, i, j)) { J->status = 1; return; }
            gold += sd[IDX(i, j, ld)];
            if (!hit[IDX(i, j, st)]) {
                hit[IDX(i, j, st)] = 1;
                mu[IDX(i, j, ld)] -= g;
            }
        }
        if (J->logZ) J->logZ[b] = lz - gold;
        return;
    }
    if (J->logZ) J->logZ[b] = lz;
    if (J->job == JOB_LOGZ || !J->mu) return;
    double *mu = J->mu + (size_t)b * blk;
    if (J->job == JOB_MARG_ADJ)
        adjoint_marginals(n, ld, c1, g, c2, tmp, mu);
    else
        outside_marginals(n, ld, sd, c1, lz, g, c2, tmp, mu);
}

static void *worker(void *arg)
{
    job_t *J = (job_t *)arg;
    const size_t st = (size_t)J->ld;           /* n+1 <= ld */
    const size_t need = st * st + 2 * st * st + 2 * st + 8;
    double *buf = (double *)malloc(need * sizeof(double));
    if (!buf) { J->status = 2; return NULL; }
    for (;;) {
        const int b = __sync_fetch_and_add(&J->next, 1);
        if (b >= J->B) break;
        run_one(J, b, buf);
    }
    free(buf);
    return NULL;
}

static int run_job(job_t *J, int nthreads)
{
    if (J->B < 0 || J->ld < 2 || !J->len || !J->s) return 1;
    for (int b = 0; b < J->B; ++b)
        if (J->len[b] < 1 || J->len[b] > J->ld - 1) return 1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    J->next = 0;
    J->status = 0;
    if (nthreads == 1) {
        worker(J);
        return J->status;
    }
    pthread_t th[256];
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, worker, J) != 0) break;
        ++started;
    }
    if (started == 0) worker(J);
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    return J->status;
}

/* ------------------------------------------------------------------------ */
/* Exported entry points.  Return 0 on success, 1 on bad arguments, 2 when
 * out of memory.  All outputs are float64 except spans (int32).           */

/* log Z per sentence (Eq. tree-prob, Algorithm 1). */
int orc_logz(int B, int ld, const int32_t *len, const float *s, double *logZ, int nthreads)
{
    job_t J = {JOB_LOGZ, B, ld, 1, len, s, NULL, logZ, NULL, NULL, NULL, 0, 0};
    return run_job(&J, nthreads);
}

/* log Z and span marginals g[b] * p((i,j)|x) (Eq. partial-derivative).
 * method 0: reverse-mode adjoint; method 1: log-space outside pass.
 * mu is [B][ld][ld]; only cells 0 <= i < j <= n_b are written.            */
int orc_marginals(int B, int ld, const int32_t *len, const float *s, const double *g,
                  double *logZ, double *mu, int method, int nthreads)
{
    if (!mu) return 1;
    job_t J = {method == 1 ? JOB_MARG_OUT : JOB_MARG_ADJ, B, ld, 1, len, s, g, logZ, mu,
               NULL, NULL, 0, 0};
    return run_job(&J, nthreads);
}

/* CKY 1-best tree: spans [B][2(ld-1)-1][2] in preorder, rows past 2n_b-1
 * set to -1; best[b] = score of that tree (may be NULL).                   */
int orc_cky(int B, int ld, const int32_t *len, const float *s, int32_t *spans, double *best,
            int nthreads)
{
    if (!spans) return 1;
    job_t J = {JOB_CKY, B, ld, 1, len, s, NULL, best, NULL, spans, NULL, 0, 0};
    return run_job(&J, nthreads);
}

/* One-stage labelled CRF: s is [B][ld][ld][L]; logZ[b]; mu (nullable) is
 * [B][ld][ld][L] with g[b] * p((i,j,l)|x).                                 */
int orc_labeled(int B, int ld, int L, const int32_t *len, const float *s, const double *g,
                double *logZ, double *mu, int nthreads)
{
    if (L < 1) return 1;
    job_t J = {JOB_LABEL, B, ld, L, len, s, g, logZ, mu, NULL, NULL, 0, 0};
    return run_job(&J, nthreads);
}

/* Gold-tree CRF loss and its gradient (Sec. 2.3, Eq. bracket-loss; Sec. 3.2):
 * gold is [B][2(ld-1)-1][2], its first 2n_b-1 rows the gold tree's spans;
 * loss[b] = log Z - s(x,y); grad is [B][ld][ld] with
 * g[b] (p((i,j)|x) - 1[(i,j) in y]) on valid cells.
 * Returns 1 if a gold row is not a span of its sentence.                   */
int orc_loss(int B, int ld, const int32_t *len, const float *s, const int32_t *gold, const double *g,
             double *loss, double *grad, int nthreads)
{
    if (!gold || !grad) return 1;
    job_t J = {JOB_LOSS, B, ld, 1, len, s, g, loss, grad, (int32_t *)gold, NULL, 0, 0};
    return run_job(&J, nthreads);
}

/* One-stage labelled decoding: s is [B][ld][ld][L]; spans [B][2(ld-1)-1][2]
 * and labels [B][2(ld-1)-1] of the best labelled tree (rows past 2n_b-1 are
 * -1); best[b] (nullable) its score.                                        */
int orc_labeled_cky(int B, int ld, int L, const int32_t *len, const float *s, int32_t *spans,
                    int32_t *labels, double *best, int nthreads)
{
    if (L < 1 || !spans || !labels) return 1;
    job_t J = {JOB_LCKY, B, ld, L, len, s, NULL, best, NULL, spans, labels, 0, 0};
    return run_job(&J, nthreads);
}

/* Labelling stage on given trees: labels[b][r] = argmax_l s(i,j,l) for every
 * row r of spans[b] that is a span of sentence b, else -1.                  */
int orc_label_spans(int B, int ld, int L, const int32_t *len, const float *s, const int32_t *spans,
                    int32_t *labels, int nthreads)
{
    if (L < 1 || !spans || !labels) return 1;
    job_t J = {JOB_LSPANS, B, ld, L, len, s, NULL, NULL, NULL, (int32_t *)spans, labels, 0, 0};
    return run_job(&J, nthreads);
}
