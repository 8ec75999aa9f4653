/*
 * switchsd_oracle.h -- plain, slow CPU oracle of SwitchSD's per-step
 * speculation-control path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes,
 * links or calls this code; only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark do.  It shares no source with the HIP
 * path: every step below is written out from the paper's definitions.
 *
 * Paper: "To Copy or Not to Copy: Controlling Speculative Decoding via
 * Intrinsic Model Signals" (SwitchSD).
 *   step 1  suffix n-gram match      -- Sec. 3.3 (Copy-Intent Decision Rule:
 *                                       kappa-gram with a prior occurrence;
 *                                       Copy-Based Speculative Generation:
 *                                       candidates ranked by recency)
 *   step 2  copy-intent probe        -- Sec. 3.2, Eq. 3 (linear, sigmoid)
 *   step 3  copy / neural switch     -- Sec. 3.3, Eq. 4 plus the kappa gate
 *   step 4  greedy verification      -- Sec. 2 (Speculative Decoding), Sec. 3.3
 *                                       (select the longest validated
 *                                       continuation), App. A (T = 0)
 *
 * All pointers are host pointers.  Arrays are contiguous, row-major.
 */
#ifndef SWITCHSD_ORACLE_H
#define SWITCHSD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_MAX_NGRAM 8

typedef struct {
    int32_t n_ngram;                      /* number of n-gram lengths tried     */
    int32_t ngram_lens[ORACLE_MAX_NGRAM]; /* tried in this order (longest first) */
    int32_t kappa;                        /* copy only if match_n >= kappa       */
    int32_t k;                            /* maximum copy-draft length (D)       */
    float theta;                          /* probe threshold as a logit          */
    int32_t n_cand;                       /* copy candidates W (0 or 1: one)     */
} oracle_cfg;

/* Step 1 for one sequence x[0..L-1] with W = max(1, n_cand) candidates.
 * Writes match_n, match_end[W] (-1 padded), copy_len[W] (0 padded) and
 * copy_tokens[W*k] (-1 padded), candidates in order of recency.  Returns the
 * number of candidates found. */
int oracle_match(const int32_t *x, int32_t L, const oracle_cfg *cfg,
                 int32_t *match_n, int32_t *match_end, int32_t *copy_len,
                 int32_t *copy_tokens);

/* Step 2 for one hidden vector: z = w . h + bias, rounded once to float. */
float oracle_probe(const uint16_t *h_bf16, const float *w, int32_t d, float bias);

/* Step 3 for one sequence.  Writes the chosen draft in node layout
 * (R rows; node 0 is the anchor); a copy draft is one chain per candidate,
 * each hanging off the anchor, candidates in order.  copy_len[W] and
 * copy_tokens[W*k] as written by oracle_match.  Returns use_copy. */
int32_t oracle_select(int32_t match_n, const int32_t *copy_len, const int32_t *copy_tokens,
                      float z, const int32_t *ntok, const int32_t *npar,
                      int32_t nn, int32_t R, const oracle_cfg *cfg,
                      int32_t *dtok, int32_t *dpar, int32_t *dn);

/* Step 4a: lowest index of the largest bf16 value of one row. */
int32_t oracle_argmax_row(const uint16_t *row_bf16, int32_t V);

/* Step 4a at T > 0 (App. A, sampling temperature).  The target's
 * distribution p = softmax(l / T) at a drafted position is realized with
 * integer weights, so that every sum and decision is exact:
 *   c   = (float)(log2(e) / T)                     (oracle_sample_scale)
 *   m   = the largest non-NaN value of the row
 *   t_j = (l_j - m) * c  in float
 *   w_j = floor(2^40 * 2^k * P(t_j - k)), k = rint(t_j), P the degree-6
 *         Taylor polynomial of 2^f, Horner in float with fused multiply-adds;
 *         0 for t_j < -41, NaN or -inf              (oracle_sample_weight)
 *   Z   = sum_j w_j (exact, 64-bit)                  (oracle_row_weights)
 *   y   = the smallest j with w_0 + ... + w_j > floor(u * Z / 2^64) for a
 *         64-bit uniform u                           (oracle_draw)
 * A row whose maximum is not finite (all NaN, -inf or +inf present) has
 * one-hot weights 2^40 at its greedy choice.  One-hot drafts (copy drafts,
 * trees, drafts without their distribution): the target's token y_r is drawn
 * at every drafted row r, and node i is accepted iff its parent is accepted
 * and its token equals y at the parent (speculative sampling with a one-hot
 * draft distribution emits tokens with the same law). */
float oracle_sample_scale(float temperature);
uint64_t oracle_sample_weight(float l, float m, float c);
uint64_t oracle_row_weights(const uint16_t *row_bf16, int32_t V, float c, uint64_t *w);
int32_t oracle_draw(const uint64_t *w, int32_t V, uint64_t Z, uint64_t u);
int32_t oracle_sample_row(const uint16_t *row_bf16, int32_t V, float c, uint64_t u);

/* Speculative sampling with the draft's own distribution q (Sec. 2; App. A),
 * for drafts that come with it (a neural chain; row r of the draft logits is
 * the draft model's output at node r, from which node r + 1 was drawn, taken
 * at the same temperature and with the same integer weights, Q_j / Zq):
 *   accept x  iff  u * Q_x * Zp < 2^64 * P_x * Zq       (oracle_spec_accept)
 * (probability min(1, p(x) / q(x)) for a uniform 64-bit u; x outside [0, V)
 * is rejected), and after a rejection the emitted token is drawn from
 *   R_j = max(0, P_j * Zq - Q_j * Zp)                   (oracle_residual_row)
 * by inverse CDF with floor(u * sum R / 2^64) (exact 128/192-bit integers). */
int32_t oracle_spec_accept(const uint16_t *p_row, const uint16_t *q_row, int32_t V, float c,
                           int32_t x, uint64_t u);
int32_t oracle_residual_row(const uint16_t *p_row, const uint16_t *q_row, int32_t V, float c,
                            uint64_t u);

/* Step 4b: accept walk over a chosen draft given the argmax of every
 * draft row.  Writes accept_len, accept_node, bonus and out_tokens[R]. */
void oracle_accept(const int32_t *dtok, const int32_t *dpar, int32_t dn,
                   const int32_t *amax, int32_t R,
                   int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                   int32_t *out_tokens);

/* Attention mask of a draft tree for the parallel verification pass:
 * bit j of row i (words of 32 bits, `words` per row) is set iff node j is
 * node i or one of its ancestors (the walk stops at an invalid parent).  Rows
 * at and beyond dn are zero. */
void oracle_tree_mask(const int32_t *dpar, int32_t dn, int32_t R, int32_t words,
                      uint32_t *mask);

/* Commit of one sequence after its step (Sec. 3.3, KV Cache Synchronization:
 * lazy propagation).  The accept_len accepted tokens and the bonus
 * (out_tokens[0..accept_len]) are appended to the context x at L =
 * clamp(*length, 0, Lmax); the context stops at Lmax (tokens past it are
 * dropped).  The draft model's cache position: after a copy step it is
 * unchanged (the draft model saw nothing new); after a neural step it is L +
 * accept_len (it drafted the accepted tokens itself; the bonus is new to it);
 * it is clamped to [0, new length].  lag = new length - draft position, the
 * tokens the next neural drafting pass must consume first. */
void oracle_commit(int32_t *x, int32_t *length, int32_t Lmax, const int32_t *out_tokens,
                   int32_t accept_len, int32_t use_copy, int32_t *draft_pos, int32_t *lag);

/* Copy-mode labels of one sequence x[0..L-1] (Sec. 3.2, Problem
 * Formulation): position j is copy-mode (labels[j] = 1) iff it lies inside a
 * window of n consecutive tokens that also occurs earlier, i.e. some window
 * x[s..s+n-1] with s <= j <= s+n-1, s+n-1 <= L-1, equals x[s'..s'+n-1] for
 * some s' < s (overlap allowed); else 0.  labels[j] = 0 for j >= L, up to
 * Lmax. */
void oracle_copy_labels(const int32_t *x, int32_t L, int32_t Lmax, int32_t n,
                        uint8_t *labels);

/* The whole step for B sequences; threads > 1 splits the batch across
 * POSIX threads (sequences are independent).  npar may be NULL (chains).
 * amax [B,R] receives the argmax of rows r < dn[b] and -1 elsewhere.
 * match_end and copy_len are [B,W], copy_tokens [B,W,k] (W = max(1, n_cand)).
 * temperature > 0 draws each row's token with oracle_sample_row and
 * uniforms[b,r] (amax then holds the drawn tokens); temperature <= 0 is the
 * greedy step and uniforms may be NULL.  draft_logits [B,R,V] (T > 0 and
 * chain drafts only, with accept_uniforms [B,R]): a sequence whose neural
 * draft is chosen is verified by speculative sampling with that q (rows tested
 * in order with accept_uniforms[b,r]; the residual or the bonus drawn with
 * uniforms[b,r] at the row where the step ends; amax[r] = the emitted token at
 * row r, -1 after it); a copy draft keeps the one-hot rule.
 * Returns 0, or -1 on a bad argument. */
int oracle_step(int32_t B, int32_t Lmax, int32_t d, int32_t R, int32_t V,
                const int32_t *tokens, const int32_t *lengths,
                const uint16_t *hidden, const float *w, float bias,
                const int32_t *ntok, const int32_t *npar, const int32_t *nn,
                const uint16_t *logits, const oracle_cfg *cfg,
                int32_t *match_n, int32_t *match_end, int32_t *copy_len,
                int32_t *copy_tokens, float *z, int32_t *use_copy,
                int32_t *dtok, int32_t *dpar, int32_t *dn, int32_t *amax,
                int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                int32_t *out_tokens, float temperature, const uint64_t *uniforms,
                const uint16_t *draft_logits, const uint64_t *accept_uniforms,
                int32_t threads);

#ifdef __cplusplus
}
#endif

#endif
