/*
 * switchsd.h -- C ABI of the SwitchSD speculation-control library (gfx950).
 *
 * Paper: "To Copy or Not to Copy: Controlling Speculative Decoding via
 * Intrinsic Model Signals".  One decoding step of SwitchSD, for B sequences:
 *
 *   1. suffix n-gram match over the token history (the copy candidates) --
 *      Sec. 3.3, Copy-Intent Decision Rule (a kappa-gram ending at the current
 *      token must have a prior occurrence) and Copy-Based Speculative
 *      Generation (up to W continuations of up to D tokens taken from the
 *      context, ranked by recency);
 *   2. linear copy-intent probe on the target's hidden state -- Sec. 3.2,
 *      Eq. 3 (p = sigmoid(w^T H), no bias in the paper; an optional bias is
 *      carried here);
 *   3. copy-versus-neural switch -- Sec. 3.3, Eq. 4 plus the kappa gate;
 *   4. greedy verification -- Sec. 2 (Speculative Decoding) and App. A
 *      (T = 0): the target's token at each drafted position is the argmax of
 *      its logits, and the longest validated continuation is kept (Sec. 3.3,
 *      Parallel Verification) together with the target's next token (bonus);
 *      at sampling temperature T > 0 the target's tokens are drawn instead
 *      (App. A; switchsd_verify_sample).
 *
 * Around the step: the verification mask of the drafts (switchsd_tree_mask),
 * the decode loop's commit with the draft model's lazy-propagation counters
 * (switchsd_commit, or `commit` in switchsd_step; Sec. 3.3, KV Cache
 * Synchronization), and the copy-mode labels the probe is trained on
 * (switchsd_copy_labels; Sec. 3.2).
 *
 * Conventions for every entry point:
 *   - All array pointers are DEVICE pointers owned by the caller; arrays are
 *     contiguous and row-major.  The library never allocates or frees.
 *   - Every call is asynchronous on `stream` and never synchronizes; outputs
 *     are valid once the caller has synchronized with the stream.
 *   - bf16 values are passed as their 16-bit patterns (uint16_t).
 *   - Token ids are int32 and only compared for equality; -1 pads outputs.
 *   - Drafts use a node layout of R rows per sequence: node 0 is the anchor
 *     (the last context token; its token field is -1, its parent -1), node i
 *     has parent dpar[i] < i.  Row r of the logits is the target's output at
 *     node r, so node i is accepted iff its parent p is accepted and
 *     dtok[i] == argmax(logits[p]).  A chain of m tokens is nodes 1..m with
 *     dpar[i] = i - 1 and dn = m + 1.
 *   - Device data is not validated, but it cannot make the library read or
 *     write out of bounds: lengths are clamped to [0, Lmax], node counts to
 *     [1, R], and a node whose parent is not in [0, i) is never accepted.
 *   - Host-side validation runs before any HIP call; on failure a negative
 *     status is returned and nothing is launched.  B = 0 is a valid no-op.
 *   - Calls that take a workspace (the step and its stages) need
 *     `switchsd_workspace_bytes(B, R, Lmax, cfg.n_cand)` bytes, 256-byte
 *     aligned, zeroed once by the caller at allocation.  Every kernel leaves
 *     the workspace zeroed again when it completes (tickets, slots, row keys,
 *     candidate lists), so no per-call clearing is needed, and calls of
 *     different shapes may share one workspace of the largest size.  After a call fails inside HIP, or if the
 *     stream is torn down mid-call, zero it again.  Calls that share one
 *     workspace must be ordered (same stream, or synchronized).
 */
#ifndef SWITCHSD_H
#define SWITCHSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t;

typedef enum {
    SWITCHSD_OK = 0,
    SWITCHSD_EINVAL = -1,    /* null pointer, bad configuration value        */
    SWITCHSD_ESHAPE = -2,    /* sizes out of range or inconsistent           */
    SWITCHSD_EHIP = -3,      /* a HIP runtime call or kernel launch failed   */
    SWITCHSD_EWORKSPACE = -4, /* workspace null, misaligned or too small     */
    SWITCHSD_EDEVICE = -5,    /* reported by switchsd_workspace_status: a
                                 bounded device-side wait gave up           */
    SWITCHSD_ESCRATCH = -6    /* switchsd_step_noalloc: the call needs more
                                 than SWITCHSD_NOALLOC_SCRATCH_BYTES         */
} switchsd_status;

#define SWITCHSD_MAX_NGRAM 8       /* most n-gram lengths in one configuration  */
#define SWITCHSD_MAX_NGRAM_LEN 64  /* longest n-gram length                     */
#define SWITCHSD_MAX_R 1024        /* most draft nodes (logits rows) per sequence */
#define SWITCHSD_MAX_CAND 16       /* most copy candidates W                     */
/* device scratch of switchsd_step_noalloc, per GPU (32 MiB)                  */
#define SWITCHSD_NOALLOC_SCRATCH_BYTES (32u << 20)

/* Step configuration.
 *   ngram_lens  lengths searched, strictly descending, each in [1, 64]; the
 *               first length with an occurrence wins, and among its
 *               occurrences the most recent one (Sec. 3.3, recency).
 *               The paper's setting is {5}; the synthetic workloads use {3,2,1}.
 *   kappa       copy is allowed only if the matched length is >= kappa
 *               (the paper's kappa = 5).  kappa >= 1.
 *   k           maximum length of one copy candidate (the paper's D = 20).
 *   n_cand      copy candidates W in [0, 16]; 0 and 1 both mean one (the
 *               paper's W = 10, Sec. 3.3 and App. D).  A copy draft holds up to
 *               W * k tokens: 1 + W * k <= R.
 *   theta       probe threshold as a logit: copy needs z >= theta, which is
 *               sigmoid(z) >= tau for theta = log(tau / (1 - tau)).
 *               -inf gives the CopySpec rule (copy iff a match exists),
 *               +inf or NaN switches copying off. */
typedef struct {
    int32_t n_ngram;
    int32_t ngram_lens[SWITCHSD_MAX_NGRAM];
    int32_t kappa;
    int32_t k;
    float theta;
    int32_t n_cand;
} switchsd_cfg;

/* Step 1 -- Sec. 3.3.  For each sequence b with L = clamp(lengths[b], 0, Lmax)
 * and context x = tokens[b, 0..L-1]: for each n in cfg->ngram_lens (in
 * order), the occurrences of the suffix x[L-n..L-1] that end at e <= L-2
 * (overlap with the suffix allowed).  The first n with an occurrence gives
 * match_n[b] = n; its W = max(1, n_cand) largest ends e_0 > e_1 > ... are the
 * candidates, most recent first: match_end[b, c] = e_c, and candidate c is
 * copy_tokens[b, c, j] = x[e_c+1+j] for j < copy_len[b, c] = min(k, L-1-e_c),
 * -1 after.  Candidate slots without an occurrence (all of them when there is
 * no match, and then match_n = 0) hold match_end = -1, copy_len = 0.
 *   tokens [B, Lmax] int32, lengths [B] int32;
 *   outputs match_n [B], match_end, copy_len [B, W] int32, copy_tokens
 *   [B, W, k] int32 (may be NULL when k == 0). */
int switchsd_ngram_match(const int32_t *tokens, const int32_t *lengths, int32_t B, int32_t Lmax,
                         const switchsd_cfg *cfg, int32_t *match_n, int32_t *match_end,
                         int32_t *copy_len, int32_t *copy_tokens, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* Step 2 -- Sec. 3.2, Eq. 3.  z[b] = sum_i h[b,i] * w[i] + bias, with every
 * product exact and the sum carried in double-double, rounded once to float.
 * The probability of copy-mode is sigmoid(z[b]).
 *   hidden [B, d] bf16 bits, w [d] float, z [B] float.  d may be 0 (z = bias). */
int switchsd_probe_score(const uint16_t *hidden, const float *w, float bias, int32_t B,
                         int32_t d, float *z, hipStream_t stream);

/* Step 3 -- Sec. 3.3, Eq. 4 and the kappa gate.
 * use_copy[b] = (match_n[b] >= kappa) && (z[b] >= theta).  The chosen draft is
 * written in node layout: copy -> the W candidates placed one after another
 * behind the anchor (Sec. 3.3, Parallel Verification), candidate c a chain of
 * its copy_len[b, c] tokens whose first node hangs off the anchor
 * (dn = 1 + sum_c copy_len[b, c]; with W = 1 the chain of the one candidate);
 * neural -> the neural draft as given (ntok/npar, with nn[b] nodes including
 * the anchor; npar == NULL means a chain).  Rows at and beyond dn[b] hold -1.
 *   match_n [B] int32, copy_len [B, W] int32 (clamped to [0, k]),
 *   copy_tokens [B, W, k] int32, z [B] float, ntok [B, R] int32,
 *   npar [B, R] int32 or NULL, nn [B] int32;
 *   outputs use_copy, dn [B] int32, dtok, dpar [B, R] int32. */
int switchsd_select_draft(const int32_t *match_n, const int32_t *copy_len,
                          const int32_t *copy_tokens, const float *z, const int32_t *ntok,
                          const int32_t *npar, const int32_t *nn, int32_t B, int32_t R,
                          const switchsd_cfg *cfg, int32_t *use_copy, int32_t *dtok,
                          int32_t *dpar, int32_t *dn, hipStream_t stream);

/* Step 4 -- Sec. 2, Sec. 3.3 (Parallel Verification), App. A (T = 0).
 * For each row r < dn[b]: amax[b,r] = the lowest index holding the largest
 * value of logits[b,r,:] (-0 equals +0, NaN is below every number, a row of
 * NaN gives 0); rows r >= dn[b] are not read and give amax = -1.  Accepted
 * nodes: node 0, and node i when its parent is accepted and
 * dtok[b,i] == amax[b,dpar[b,i]].  accept_node[b] = the deepest accepted node
 * (ties to the lowest index), accept_len[b] = its depth,
 * bonus[b] = amax[b, accept_node[b]], out_tokens[b, :] = the accepted path
 * tokens (anchor excluded), then the bonus, then -1.
 *   logits [B, R, V] bf16 bits (2-byte aligned), dtok/dpar [B, R], dn [B];
 *   dpar == NULL means chains; amax [B, R] may be NULL. */
int switchsd_verify_accept(const uint16_t *logits, int32_t B, int32_t R, int32_t V,
                           const int32_t *dtok, const int32_t *dpar, const int32_t *dn,
                           int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                           int32_t *out_tokens, int32_t *amax, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* Step 4 at sampling temperature T > 0 -- App. A (throughput at T > 0 with
 * speculative sampling).  The target's distribution at drafted row r is
 * p_r = softmax(logits[b,r,:] / T), realized with integer weights
 *   w_j = floor(2^40 * 2^k P(t_j - k)),  t_j = (l_j - m) * c  (float),
 *   c = (float)(log2(e) / T), m = the largest non-NaN value of the row,
 *   k = rint(t_j), P the degree-6 Taylor polynomial of 2^f evaluated by
 *   Horner's rule in fused multiply-adds,
 * which are 0 for t_j < -40.5 (and for NaN and -inf).  A row without a finite
 * maximum (every value NaN, -inf, or +inf present) has one-hot weights at its
 * greedy choice.  The normalized weights are within total variation 1e-6 of
 * the exact softmax at vocabularies up to 151936 (measured <= 1e-7).  A draw
 * with the 64-bit uniform u is the smallest j with w_0 + ... + w_j >
 * floor(u * Z / 2^64), Z = sum_j w_j: the sums are exact integers, so y does
 * not depend on the order of the reduction.
 * The drafts are tokens (copy candidates are deterministic; neural drafts come
 * without their distribution), so the draft distribution is one-hot and
 * speculative sampling (accept x with probability p(x)/q(x), else draw from
 * the normalized residual max(0, p - q)) emits the same token law as: draw
 * y_r from p_r with uniforms[b,r] for every drafted row r < dn[b], accept node
 * i iff its parent is accepted and dtok[b,i] == y_{parent}.  The accept result
 * is then formed exactly as in switchsd_verify_accept with y in place of the
 * argmax (amax[b,r] = y_r).
 * Drafts that come with their distribution q (draft_logits != NULL; chains
 * only, dpar == NULL): row r of draft_logits holds the draft model's logits
 * at node r, from which node r + 1 was drawn; q_r = softmax(draft_logits[b,r]
 * / T) with the same integer weights (Q_j / Zq, p_r being P_j / Zp).  This is
 * speculative sampling proper (Sec. 2): rows r = 0, 1, ... are tested in
 * order, node r + 1 with token x being accepted iff
 *   accept_uniforms[b,r] * Q_x * Zp < 2^64 * P_x * Zq
 * (probability min(1, p(x)/q(x)); x outside [0, V) is rejected); at the first
 * rejected row a the emitted token is drawn with uniforms[b,a] from the
 * residual R_j = max(0, P_j * Zq - Q_j * Zp) (from p if the residual is empty),
 * and with no rejection the bonus is drawn from p at row dn - 1.  Then
 * accept_len = accept_node = a, out_tokens = the accepted tokens and the
 * emitted one, amax[b,r] = the token emitted at row r (-1 after a).  The
 * emitted tokens follow p exactly up to the weights' error and the uniforms'
 * 2^-64 resolution.
 *   temperature > 0 and finite; uniforms [B, R] uint64 (only rows r < dn[b]
 *   are read); accept_uniforms [B, R] uint64 (with draft_logits, else
 *   ignored); logits and draft_logits [B, R, V] bf16 bits, 16-byte aligned,
 *   V % 8 == 0 and V <= 524288; sample_workspace of
 *   switchsd_sample_workspace_bytes(B, R, V) bytes, 256-byte aligned, no
 *   initialization needed; other arguments as in switchsd_verify_accept.
 *   Launches: the row maxima, then the weight sums, in which one work-group per
 *   row draws the row's token (without q, R <= 64 and B * R no larger than the
 *   compute-unit count: the row's first, polling the others' sums; else the
 *   last to arrive); with q the first launch also takes the q row maxima (a
 *   launch of their own for streamed long drafts), the weight sums take the
 *   accept tests, and the residual draw comes last. */
int switchsd_verify_sample(const uint16_t *logits, int32_t B, int32_t R, int32_t V,
                           float temperature, const uint64_t *uniforms,
                           const uint16_t *draft_logits, const uint64_t *accept_uniforms,
                           const int32_t *dtok, const int32_t *dpar, const int32_t *dn,
                           int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                           int32_t *out_tokens, int32_t *amax, void *workspace,
                           size_t workspace_bytes, void *sample_workspace,
                           size_t sample_workspace_bytes, hipStream_t stream);

/* Bytes of the scratch a draw at T > 0 needs (the weight sums per 16 KB chunk
 * and wave of every row). */
size_t switchsd_sample_workspace_bytes(int32_t B, int32_t R, int32_t V);

/* Attention mask of the chosen drafts for the target's verification pass --
 * Sec. 3.3, Parallel Verification with Block-Triangular Attention: a drafted
 * token attends to the whole prefix (not represented here) and to the draft
 * nodes on its own path back to the anchor, itself included; for W copy
 * candidates this is block-triangular (each candidate sees only its own
 * earlier tokens).  mask[b, i, :] is a bitset of words = (R + 31) / 32 uint32
 * words: bit j of word j / 32 is set iff node j is node i or one of its
 * ancestors, the walk stopping at a parent outside [0, node).  Rows
 * i >= clamp(dn[b], 0, R) are all zero.
 *   dpar [B, R] int32 or NULL (chains), dn [B] int32;
 *   output mask [B, R, (R + 31) / 32] uint32. */
int switchsd_tree_mask(const int32_t *dpar, const int32_t *dn, int32_t B, int32_t R,
                       uint32_t *mask, hipStream_t stream);

/* How switchsd_step schedules its work. */
typedef enum {
    SWITCHSD_MODE_AUTO = 0,  /* FUSED when every row may be needed (1 + W k >= R) and
                                R <= 64, else SPLIT                                       */
    SWITCHSD_MODE_FUSED = 1, /* one launch; reads rows r < max(nn[b], 1 + W k)                */
    SWITCHSD_MODE_SPLIT = 2  /* two launches; reads only rows r < dn[b] of the chosen draft  */
} switchsd_mode;

/* All arguments of one step (steps 1-4 in order).  Inputs as in the stage
 * calls above; every output pointer is required except amax. */
typedef struct {
    const int32_t *tokens;   /* [B, Lmax] */
    const int32_t *lengths;  /* [B]       */
    const uint16_t *hidden;  /* [B, d] bf16 bits */
    const float *w;          /* [d]       */
    const int32_t *ntok;     /* [B, R] neural draft tokens */
    const int32_t *npar;     /* [B, R] neural draft parents, NULL = chains */
    const int32_t *nn;       /* [B] neural draft node count (anchor included) */
    const uint16_t *logits;  /* [B, R, V] bf16 bits */
    int32_t B, Lmax, d, R, V;
    float bias;
    switchsd_cfg cfg;
    int32_t mode;            /* switchsd_mode */
    int32_t *match_n, *match_end, *copy_len, *copy_tokens; /* [B],[B,W],[B,W],[B,W,k] */
    float *z;                                              /* [B] */
    int32_t *use_copy, *dtok, *dpar, *dn;                  /* [B],[B,R],[B,R],[B] */
    int32_t *amax;                                         /* [B, R] or NULL */
    int32_t *accept_len, *accept_node, *bonus, *out_tokens; /* [B],[B],[B],[B,R] */
    /* T > 0 (switchsd_verify_sample); 0 for the greedy step (the fields below
     * are then unused) */
    float temperature;
    const uint64_t *uniforms;  /* [B, R] */
    void *sample_workspace;
    size_t sample_workspace_bytes;
    /* decode loop: commit != 0 appends the accepted tokens and the bonus to
     * tokens/lengths in the same launch (they are then read-write) and
     * updates draft_pos and lag as switchsd_commit does */
    int32_t commit;
    int32_t *draft_pos;      /* [B] in/out */
    int32_t *lag;            /* [B] out    */
    /* T > 0 with the neural draft's own distribution (switchsd_verify_sample's
     * draft_logits; NULL = one-hot drafts): a sequence whose neural draft is
     * chosen is verified by speculative sampling with it, a copy draft keeps
     * the one-hot rule.  Needs npar == NULL (chains). */
    const uint16_t *draft_logits;     /* [B, R, V] bf16 bits */
    const uint64_t *accept_uniforms;  /* [B, R] */
} switchsd_step_args;

/* One whole step.  Results are identical to calling the four stage entry
 * points in order (switchsd_verify_sample as step 4 when temperature != 0);
 * MODE_FUSED does the greedy step in one kernel launch. */
int switchsd_step(const switchsd_step_args *args, void *workspace, size_t workspace_bytes,
                  hipStream_t stream);

/* switchsd_step for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Identical results to switchsd_step; the workspace and the scratch of a draw
 * at T > 0 (args->sample_workspace is ignored) come from a fixed device array
 * of SWITCHSD_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends.
 * Nothing is allocated or freed.  The array's address is looked up at the
 * first call on each GPU (with that GPU current), and that call also clears
 * the array with a kernel on `stream`, ordered before its own kernels; every
 * kernel leaves the workspace part zeroed again.  All calls on one GPU share
 * the array: calls that overlap in time (different streams, or host threads
 * without ordering) race and give undefined results.  A call that fails
 * inside HIP can leave the array dirty for the next one.
 * Returns SWITCHSD_ESCRATCH (and launches nothing) when
 * switchsd_workspace_bytes(B, R, Lmax, cfg.n_cand) rounded up to 256 bytes,
 * plus switchsd_sample_workspace_bytes(B, R, V) at T != 0, exceeds the array;
 * otherwise the codes of switchsd_step. */
int switchsd_step_noalloc(const switchsd_step_args *args, hipStream_t stream);

/* Decode-loop commit of a finished step -- Sec. 3.3, KV Cache
 * Synchronization (lazy propagation).  For each sequence, with
 * L = clamp(lengths[b], 0, Lmax) and a = clamp(accept_len[b], 0, R - 1): the
 * accepted tokens and the bonus out_tokens[b, 0..a] are appended at
 * tokens[b, L..], cut at Lmax; lengths[b] = min(L + a + 1, Lmax).  The draft
 * model's cache position draft_pos[b] stays after a copy step (the draft model
 * saw nothing new) and becomes L + a after a neural step (it drafted the
 * accepted tokens; the bonus is new to it), clamped to [0, lengths[b]];
 * lag[b] = lengths[b] - draft_pos[b] is the number of tokens the next neural
 * drafting pass must consume first.
 *   tokens [B, Lmax], lengths, draft_pos [B] int32 in/out; out_tokens [B, R],
 *   accept_len, use_copy [B] int32 in; lag [B] int32 out. */
int switchsd_commit(int32_t *tokens, int32_t *lengths, int32_t B, int32_t Lmax,
                    const int32_t *out_tokens, int32_t R, const int32_t *accept_len,
                    const int32_t *use_copy, int32_t *draft_pos, int32_t *lag,
                    hipStream_t stream);

/* Copy-mode labels for training the copy-intent probe -- Sec. 3.2, Problem
 * Formulation: position j of sequence b (L = clamp(lengths[b], 0, Lmax)) is
 * copy-mode, labels[b, j] = 1, iff it lies inside a verbatim span of at least
 * n tokens that appears earlier in the context, i.e. some window
 * x[s..s+n-1] with s <= j <= s+n-1 <= L-1 equals x[s'..s'+n-1] for some
 * s' < s (overlap allowed); 0 otherwise and for j >= L.  The paper's setting
 * is n = 5.  Offline (whole sequences, not per decoding step).
 *   tokens [B, Lmax] int32, lengths [B] int32, 1 <= n <= 64,
 *   Lmax <= 2^28; output labels [B, Lmax] uint8; workspace of
 *   switchsd_label_workspace_bytes(B, Lmax) bytes (a table of the distinct
 *   windows per sequence), 256-byte aligned, zeroed once by the caller (left
 *   zeroed by every call).  Three launches; expected time linear in
 *   B * Lmax * n. */
int switchsd_copy_labels(const int32_t *tokens, const int32_t *lengths, int32_t B, int32_t Lmax,
                         int32_t n, uint8_t *labels, void *workspace, size_t workspace_bytes,
                         hipStream_t stream);
/* 0 for a negative argument or Lmax > 2^28. */
size_t switchsd_label_workspace_bytes(int32_t B, int32_t Lmax);

/* Workspace bytes needed by calls with B sequences of R rows, contexts of up
 * to Lmax tokens and n_cand copy candidates (pass 0 for what a call does not
 * take: R for the match stage, Lmax for verification).  0 for a negative
 * argument. */
size_t switchsd_workspace_bytes(int32_t B, int32_t R, int32_t Lmax, int32_t n_cand);

/* Device-side status of the calls that used `workspace` (B sequences),
 * written to *status (a DEVICE int32) asynchronously on `stream`:
 * SWITCHSD_OK, or SWITCHSD_EDEVICE when a bounded wait inside a kernel gave
 * up since the last status call.  There are four such waits, and in
 * practice each always ends, since what it waits for was dispatched before it
 * or waits for nothing:
 *   - with contexts longer than 1024 tokens, the scan work-group that finishes
 *     a sequence's front in switchsd_step waits for the probe's work-group
 *     (dispatched before it); if it gives up, that sequence's switch takes
 *     the neural draft;
 *   - with contexts of 2 to 64 tiles of 1024 tokens and B no larger than
 *     the device's compute-unit count, the last scan tile of a sequence
 *     waits for the other tiles' match results (the tiles wait for nothing);
 *     if it gives up, a missing tile counts as holding no occurrence;
 *   - at T = 0 with R <= 64 and B no larger than the device's compute-unit
 *     count, in switchsd_step's fused launch (one candidate) and in the
 *     verification launch (switchsd_verify_accept, and switchsd_step's split
 *     mode), the work-group holding a sequence's draft waits for the results
 *     of that sequence's argmax work-groups (which wait for nothing); if it
 *     gives up, a segment whose result is missing counts as holding no
 *     maximum;
 *   - at T > 0 without draft_logits, with R <= 64 and B * R no larger than
 *     the compute-unit count, the weight-sum launch's first work-group of
 *     each row waits for the row's other sum work-groups (which wait for
 *     nothing), and row 0's then for the other rows' drawn tokens; if it
 *     gives up, a row whose sums are missing keeps its greedy choice and a
 *     missing drawn token counts as none.
 * After a give-up that sequence's outputs are not valid.  The call reads and
 * clears the error words; after SWITCHSD_EDEVICE, zero the workspace again
 * before its next use.
 *   workspace of at least switchsd_workspace_bytes(B, 0, 0, 0) bytes, the
 *   same B as the calls; status [1] int32 on the device. */
int switchsd_workspace_status(void *workspace, size_t workspace_bytes, int32_t B,
                              int32_t *status, hipStream_t stream);

/* Test support only: while `on` is nonzero, switchsd_step's probe work-groups
 * withhold their flag and the wait above gives up after a few iterations, so
 * that a test can force the give-up path (every kernel still exits). */
void switchsd_test_withhold_probe_flag(int32_t on);

/* Test support only: while `on` is nonzero, in the fused switchsd_step the
 * argmax work-group of sequence 0, row 0, first segment withholds its result
 * (at T > 0 with the polled draw: the weight-sum work-group of that segment
 * withholds its sums), and so does sequence 0's first scan tile when a context
 * has 2 to 64 tiles of 1024 tokens; the polls that wait for them give up after
 * a few iterations (every kernel still exits). */
void switchsd_test_withhold_segment(int32_t on);

/* Static, thread-safe text of a status code. */
const char *switchsd_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif
