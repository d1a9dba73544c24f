/*
 * crf_inside.h -- C ABI of the MI355X (gfx950) batched tree-CRF library.
 *
 * Method: Zhang, Zhou & Li, "Fast and Accurate Neural CRF Constituency
 * Parsing" (IJCAI 2020).  For every sentence of a batch, given span scores
 * s(i,j), the library computes
 *   - log Z(x), the log partition function over all binary bracketings
 *     (Sec. 2.1, Eq. tree-prob), by the inside recursion of Sec. 3.1
 *     (Algorithm 1);
 *   - the span marginals p((i,j)|x) = d log Z / d s(i,j) (Sec. 3.2,
 *     Eq. partial-derivative), evaluated as exp(inside + outside - log Z)
 *     with the outside recursion run beside the inside one;
 *   - the 1-best tree argmax_y s(x,y) (Sec. 2.1, Eq. tree-argmax) by CKY,
 *     the same recursion with max in place of sum (Sec. 3.3);
 *   - for the one-stage labelled CRF (Sec. 4.2, Eq. tree-label-score),
 *     log Z, the per-label span marginals p((i,j,l)|x) and the best
 *     labelled tree;
 *   - MBR decoding over the marginals (Sec. 3.3), the gold-tree CRF loss
 *     and its gradient (Sec. 2.3, Eq. bracket-loss), and the labelling stage
 *     of the two-stage parser (Sec. 2.1, Eq. label-argmax);
 *   - the span (and label) scores themselves, from boundary representations
 *     by the biaffine scorer (Sec. 2.2, Eq. biaffine).
 *
 * Conventions
 *   Fence posts.  A sentence of n words has boundaries 0..n; span (i,j),
 *   0 <= i < j <= n, covers words i..j-1 (the paper's inclusive (i, j-1)).
 *   Every legal tree contains all n width-1 spans and the root (0,n) and has
 *   2n-1 spans in all (Sec. 2.1; Fig. 1b); width-1 spans are scored.
 *
 *   Layout.  scores is float32, row-major [B][N1][N1] (unlabelled) or
 *   [B][N1][N1][L] (labelled), N1 = the padded side (>= max length + 1).
 *   s(i,j) of sentence b is scores[(b*N1 + i)*N1 + j] (times L, plus l, when
 *   labelled).  Only cells 0 <= i < j <= n_b are read; every other cell may
 *   hold anything, NaN included.  marginals has the layout of scores and only
 *   its valid cells are written: the rest of the buffer is left untouched.
 *   Outputs are in the caller's sentence order.
 *
 *   Memory.  Every float/int pointer passed to a compute call is device memory
 *   owned by the caller; the library never frees it.  lengths_host in
 *   crf_plan_create is host memory, read only during the call.  The plan owns
 *   its device copies of the lengths and schedule, a workspace for
 *   sentences whose chart does not fit in LDS and, with such sentences, a
 *   257 KB area for the teams below; they are allocated by crf_plan_create
 *   and freed by crf_plan_destroy.  Compute calls allocate nothing.
 *
 *   Teams.  When a call has only a few workspace sentences (at most 32
 *   sentence passes in one launch), each pass runs on a team of 8 or 16
 *   workgroups of one XCD that wait for each other at every width step.
 *   Such a launch waits until all its workgroups are resident at once (it
 *   is sized to fit an otherwise idle device); work from other streams
 *   delays it.  A wait that lasts about 2^21 polls (a second or two) ends
 *   the launch, and the outputs of its workspace sentences are invalid: log
 *   Z and best score NaN when a width step's wait ran out, left unwritten
 *   when the launch's workgroups never were resident together.  Two plans' team launches running at once on different streams
 *   can hold each other's room that way: issue calls that may form teams on
 *   one stream, or create the plans with CRF_NO_TEAMS.  Results are
 *   bit-identical to those of one workgroup per pass.
 *
 *   Streams.  `stream` is a hipStream_t (NULL = the null stream).  Compute
 *   calls only enqueue work and never synchronise.  Calls on one plan must
 *   not overlap on the device: issue them on one stream, or order them with
 *   events.  A plan owns device state that its calls use while they run --
 *   the fused launches' work counter, the workspace that holds the charts
 *   and CKY split tables of sentences too long for LDS (crf_plan_info:
 *   workspace_users) and the team area -- and two overlapping calls would
 *   share it.  Different
 *   plans share nothing and may run concurrently on any streams (but see
 *   Teams below for calls with a few workspace sentences).
 *
 *   Errors.  Every call returns a status (CRF_OK = 0).  Arguments are checked
 *   on the host before any HIP call is made, so a rejected call has no effect
 *   on the device.  crf_last_error() gives a message for the last failure on
 *   the calling thread.  Scores must be finite inside the valid region; NaN
 *   or infinities there give unspecified (but memory-safe) results.
 */
#ifndef CRF_INSIDE_H
#define CRF_INSIDE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    CRF_OK = 0,
    CRF_EINVAL = 1,        /* bad argument: null pointer, size or length out of range */
    CRF_ENOMEM = 2,        /* host or device allocation failed (crf_plan_create only) */
    CRF_EHIP = 3,          /* HIP runtime or launch error (see crf_last_error) */
    CRF_EUNSUPPORTED = 4   /* valid but not implemented, e.g. decode of labelled scores */
};

#define CRF_MAX_LEN 1023      /* longest sentence, in words */
#define CRF_MAX_LABELS 4096   /* most labels per span */

/* Plan flags. */
#define CRF_FORCE_SPILL 0x1u  /* run every sentence on the workspace-chart kernels */
#define CRF_NO_TEAMS 0x2u     /* one workgroup per workspace sentence pass, never teams */

typedef struct crf_plan crf_plan;

typedef struct {
    int32_t batch;           /* B */
    int32_t n1;              /* padded side N1 */
    int32_t num_labels;      /* L (1 = unlabelled) */
    int32_t max_len;         /* longest sentence */
    int32_t lds_count;       /* sentences whose inside chart lives in LDS */
    int32_t spill_count;     /* sentences whose inside chart lives in the workspace */
    int64_t workspace_bytes; /* device workspace owned by the plan */
    int32_t lds_bytes_inside;/* dynamic LDS per workgroup, inside kernels */
    int32_t lds_bytes_cky;   /* dynamic LDS per workgroup, CKY kernel */
    int32_t cky_spill_count; /* sentences whose CKY chart lives in the workspace */
    int32_t split_ws_count;  /* sentences whose CKY chart is in LDS but whose
                                split table is in the workspace */
    int32_t workspace_users; /* sentences that use the workspace in some call
                                (any of the three above) */
    int32_t fused_queue;     /* 1 if the fused launches pull work from the
                                plan's counter */
    int32_t mbr_fused;       /* 1 if crf_mbr_decode runs as one launch per
                                bundle queue (else as separate launches) */
} crf_plan_stats;

/*
 * crf_plan_create -- validate a batch shape and build its schedule.
 *   out          receives the plan (set to NULL on failure).
 *   lengths_host host int32[batch]: sentence lengths n_b, 1 <= n_b <= n1-1.
 *   batch        B >= 1.
 *   n1           padded side of the score block, 2 <= n1 <= CRF_MAX_LEN+1.
 *   num_labels   L, 1 <= L <= CRF_MAX_LABELS; 1 = unlabelled scores.
 *   flags        0, or CRF_FORCE_SPILL and/or CRF_NO_TEAMS.
 * Uses the current HIP device; later calls must run with that device current.
 * Returns CRF_EINVAL (nothing allocated), CRF_ENOMEM or CRF_EHIP.
 */
int crf_plan_create(crf_plan **out, const int32_t *lengths_host, int32_t batch, int32_t n1,
                    int32_t num_labels, uint32_t flags);

/* Free a plan and its device memory (NULL is accepted).  Synchronises the
 * device first so that no enqueued call still uses it. */
int crf_plan_destroy(crf_plan *plan);

/* Sizes and schedule summary of a plan (host only, no HIP call). */
int crf_plan_info(const crf_plan *plan, crf_plan_stats *out);

/*
 * crf_inside_fwd -- log partition function (Sec. 2.1, Eq. tree-prob; Sec. 3.1,
 * Algorithm 1).
 *   scores  device float32, layout above.
 *   logZ    device float32[B]: log Z(x_b).
 */
int crf_inside_fwd(const crf_plan *plan, const float *scores, float *logZ, void *stream);

/*
 * crf_inside_bwd -- span marginals as the gradient of log Z (Sec. 3.2,
 * Eq. partial-derivative).  The inside chart is recomputed on chip.
 *   grad_logZ  device float32[B] upstream gradient, or NULL for all ones.
 *   marginals  device float32, layout of scores: grad_logZ[b] * p((i,j)|x_b)
 *              (labelled: grad_logZ[b] * p((i,j,l)|x_b)) on valid cells only.
 */
int crf_inside_bwd(const crf_plan *plan, const float *scores, const float *grad_logZ,
                   float *marginals, void *stream);

/* crf_inside_fwd_bwd -- both of the above in one pass over the chart.
 * logZ may be NULL. */
int crf_inside_fwd_bwd(const crf_plan *plan, const float *scores, const float *grad_logZ,
                       float *logZ, float *marginals, void *stream);

/*
 * crf_cky_decode -- 1-best unlabelled tree (Sec. 2.1, Eq. tree-argmax) by CKY
 * (Sec. 3.3).  The chart is float64: beta(i,i+1) = s(i,i+1),
 * beta(i,j) = (max_k (beta(i,k) + beta(k,j))) + s(i,j); among equal maxima
 * the lowest split k is kept.
 *   spans  device int32[B][2*(N1-1)-1][2]: the 2n_b-1 spans (i,j) of the tree
 *          in preorder (i ascending, then j descending), then rows of -1.
 *   best   device float32[B] score of that tree, or NULL.
 * Unlabelled plans only (CRF_EUNSUPPORTED otherwise).
 */
int crf_cky_decode(const crf_plan *plan, const float *scores, int32_t *spans, float *best,
                   void *stream);

/*
 * crf_inside_fwd_bwd_cky -- crf_inside_fwd_bwd and crf_cky_decode in one
 * launch, their workgroups interleaved so the two run concurrently.  Same
 * arguments and results as the two calls (logZ and best may be NULL).
 * Unlabelled plans only (CRF_EUNSUPPORTED otherwise).
 */
int crf_inside_fwd_bwd_cky(const crf_plan *plan, const float *scores, const float *grad_logZ,
                           float *logZ, float *marginals, int32_t *spans, float *best,
                           void *stream);

/*
 * crf_mbr_decode -- MBR decoding (Sec. 3.3, "Decoding"): the CKY tree with the
 * span marginals p((i,j)|x) in place of the span scores in Eq. tree-score and
 * Eq. tree-argmax, i.e. the tree whose spans' marginals sum highest.  One
 * pass: the inside and outside sweeps write the marginals, and the same
 * workgroup then runs CKY over them (float64 chart, lowest split on ties, as
 * crf_cky_decode) while its bundle is still on chip.
 *   logZ       device float32[B] or NULL: log Z(x_b).
 *   marginals  device float32, layout of scores (required, must not alias
 *              scores): p((i,j)|x_b) on valid cells; the trees are decoded
 *              from exactly these float32 values.
 *   spans      device int32[B][2*(N1-1)-1][2], as crf_cky_decode.
 *   best       device float32[B] or NULL: the sum of the marginals over the
 *              tree (float64 chart, rounded).
 * Unlabelled plans only (CRF_EUNSUPPORTED otherwise).
 */
int crf_mbr_decode(const crf_plan *plan, const float *scores, float *logZ, float *marginals, int32_t *spans,
                   float *best, void *stream);

/*
 * crf_gold_loss -- the sentence-level CRF loss of a gold tree (Sec. 2.3,
 * Eq. bracket-loss), L = log Z(x) - s(x,y), with s(x,y) the sum of the gold
 * spans' scores (Eq. tree-score), and its gradient with respect to the scores,
 * dL/ds(i,j) = p((i,j)|x) - 1[(i,j) in y] (the marginals of Sec. 3.2 minus
 * the gold indicator).
 *   gold_spans  device int32[B][2*(N1-1)-1][2]: the first 2n_b-1 rows of
 *               sentence b are its gold tree's spans (i,j) (the layout
 *               crf_cky_decode writes; any order).  Rows that are not spans
 *               of the sentence (0 <= i < j <= n_b) are skipped; a repeated
 *               span adds its score to s(x,y) again but 1 to the indicator.
 *   grad_loss   device float32[B] upstream gradient dOut/dL, or NULL for 1.
 *   loss        device float32[B]: L (not scaled by grad_loss).
 *   grad_scores device float32, layout of scores (must not alias scores):
 *               grad_loss[b] * (p((i,j)|x_b) - 1[(i,j) in y_b]) on valid cells
 *               only.
 * Unlabelled plans only (CRF_EUNSUPPORTED otherwise).
 */
int crf_gold_loss(const crf_plan *plan, const float *scores, const int32_t *gold_spans, const float *grad_loss,
                  float *loss, float *grad_scores, void *stream);

/*
 * crf_cky_decode_labeled -- one-stage labelled decoding (Sec. 4.2,
 * Eq. tree-label-score; Sec. 2.1, time-complexity paragraph): the labelled
 * tree maximising the sum of s(i,j,l) over its labelled spans.  Each span's
 * label is free, so this is CKY (as crf_cky_decode) over the float32 maxima
 * max_l s(i,j,l), each of the tree's spans labelled with the lowest label
 * attaining its maximum.
 *   scores  device float32 [B][N1][N1][L], L = the plan's num_labels.
 *   spans   device int32[B][2*(N1-1)-1][2], as crf_cky_decode.
 *   labels  device int32[B][2*(N1-1)-1]: the label of each span row, -1 on
 *           the rows past the tree.
 *   best    device float32[B] or NULL: the labelled tree's score.
 */
int crf_cky_decode_labeled(const crf_plan *plan, const float *scores, int32_t *spans, int32_t *labels, float *best,
                           void *stream);

/*
 * crf_label_spans -- the labelling stage of the two-stage parser (Sec. 2.1,
 * Eq. label-argmax): every span (i,j) of a given tree independently takes
 * argmax_l s(i,j,l) (the lowest such label on ties).
 *   label_scores  device float32 [B][N1][N1][num_labels] (N1 and B of the
 *                 plan; the plan's own num_labels is not used).
 *   num_labels    1 <= num_labels <= CRF_MAX_LABELS.
 *   spans         device int32[B][2*(N1-1)-1][2], e.g. crf_cky_decode's or
 *                 crf_mbr_decode's output.
 *   labels        device int32[B][2*(N1-1)-1]: the label of every row that is
 *                 a span of its sentence (0 <= i < j <= n_b), else -1.
 */
int crf_label_spans(const crf_plan *plan, const float *label_scores, int32_t num_labels, const int32_t *spans,
                    int32_t *labels, void *stream);

/*
 * crf_biaffine_scores -- the biaffine span scorer that produces the span
 * scores (Sec. 2.2, Eq. biaffine): s(i,j) = [r^l_i ; 1]^T W r^r_j from the
 * left boundary representation of fence post i and the right one of fence
 * post j, W of (d+1) x d entries (the appended 1 makes its last row a bias on
 * r^r_j); one W per label for label scores (Sec. 2.2, label scoring):
 * s(i,j,l) = [r^l_i ; 1]^T W_l r^r_j.  bf16 inputs, fp32 products and sums
 * on the matrix cores (MFMA); the inner (d x d) product stays on chip.
 *   rl, rr      device bf16 bit patterns [B][N1][d]: r^l_i and r^r_i of
 *               sentence b at [(b*N1 + i)*d]; rows past n_b are not read.
 *               8-byte aligned.
 *   w           device bf16 bit patterns [num_labels][d][ldw], W transposed:
 *               w[(l*d + c)*ldw + a] = W_l[a][c] for a <= d (a = d is the bias
 *               row); entries a > d are not read.  8-byte aligned.
 *   d           4 <= d <= 508, a multiple of 4 (the paper's d is 500, and
 *               100 for the label scorer).
 *   ldw         row stride of w, >= d+1 and a multiple of 4.
 *   num_labels  number of W (1 for span scores).
 *   scores      device float32, [B][N1][N1] when num_labels = 1 (the layout
 *               the CRF calls take), else [B][N1][N1][num_labels]; only cells
 *               0 <= i < j <= n_b are written.
 * B, N1 and the lengths are the plan's (its own num_labels is not used).
 */
int crf_biaffine_scores(const crf_plan *plan, const uint16_t *rl, const uint16_t *rr, const uint16_t *w,
                        int32_t d, int32_t ldw, int32_t num_labels, float *scores, void *stream);

/*
 * crf_inside_fwd_bwd_cky_noalloc -- crf_inside_fwd_bwd_cky for callers that
 * cannot allocate device memory or must not touch the plan's device state
 * while they run (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments and results as
 * crf_inside_fwd_bwd_cky; the plan's workspace and work counter are not
 * used: the call takes them from a static scratch array of the library,
 * 8 MiB per GPU, held from the library's first use on a device until the
 * process ends.  It calls no allocation routine; it enqueues a small kernel
 * that clears the array's counter, then the launches of the fused call
 * (with one workgroup per workspace sentence pass: no teams).
 *   Returns CRF_EINVAL when the plan needs more workspace than the array
 *   holds (8 MiB less 256 bytes; crf_plan_info: workspace_bytes), e.g. a
 *   batch with many sentences longer than 142 words.
 *   Every such call on one GPU shares that GPU's array, whatever the plan:
 *   calls of this entry point that overlap on one GPU race (issue them on
 *   one stream, or order them with events).
 */
int crf_inside_fwd_bwd_cky_noalloc(const crf_plan *plan, const float *scores, const float *grad_logZ,
                                   float *logZ, float *marginals, int32_t *spans, float *best,
                                   void *stream);

/* Static description of a status code. */
const char *crf_status_string(int status);

/* Message for the last failing call on this thread ("" if none). */
const char *crf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CRF_INSIDE_H */
