/*
 * switchsd_oracle.c -- plain, slow CPU oracle of SwitchSD's per-step
 * speculation-control path.  TEST INFRASTRUCTURE ONLY (see the header).
 *
 * Every function is the definition written out with scalar loops, in the
 * order the paper states the method.  No blocking, no packing, no early
 * exits beyond what the definition itself implies.
 *
 * Readings taken where the paper is silent (each also listed in the design
 * notes of the repository):
 *   R1  a prior occurrence may overlap the current suffix; its end e must be
 *       <= L-2 so that at least one continuation token exists;
 *   R2  the n-gram lengths are tried longest first, and among the occurrences
 *       of one length the most recent (largest end) wins -- "ranked by
 *       recency", Sec. 3.3;
 *   R3  the kappa gate is separate from the lengths searched: copy needs
 *       match_n >= kappa;
 *   R4  the threshold test PR(H) >= tau of Eq. 4 is taken in logit space as
 *       z >= theta with theta = logit(tau), in float;
 *   R5  the probe keeps an optional bias (Eq. 3 has none: bias = 0);
 *   R6  argmax ties go to the lowest vocabulary index, -0 equals +0 and NaN
 *       is below every number (a row of NaN gives index 0);
 *   R7  node 0 of a draft is the anchor; a node whose parent index is not in
 *       [0, i) is never accepted; among accepted nodes the deepest wins, ties
 *       to the lowest node index;
 *   R8  lengths are clamped to [0, Lmax] and neural node counts to [1, R];
 *   R13 W candidates are the W largest ends of the matched length, most
 *       recent first; each is its own chain behind the anchor (no merging of
 *       equal prefixes); empty slots add no nodes;
 *   R14 among equally deep accepted nodes the lowest index wins, i.e. the
 *       most recent candidate;
 *   R15 the verification mask covers draft nodes only (the prefix, seen by
 *       every drafted token, is implied); a walk stops at an invalid parent.
 */
#include "switchsd_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* bf16 is the upper half of an IEEE binary32: widening is exact. */
static float bf16_to_float(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static int32_t n_cand_of(const oracle_cfg *cfg)
{
    return cfg->n_cand > 1 ? cfg->n_cand : 1;
}

/* Step 1 -- Sec. 3.3 (Copy-Intent Decision Rule; Copy-Based Speculative
 * Generation).  For each n in the configured order: the set of ends e with
 * n-1 <= e <= L-2 and x[e-t] == x[L-1-t] for every t < n.  The first n whose
 * set is non-empty gives match_n = n.  Its W largest ends, most recent first,
 * are the candidates ("ranked by recency"); each candidate is the
 * continuation after its occurrence, cut to k tokens and to the end of the
 * context. */
int oracle_match(const int32_t *x, int32_t L, const oracle_cfg *cfg,
                 int32_t *match_n, int32_t *match_end, int32_t *copy_len,
                 int32_t *copy_tokens)
{
    const int32_t W = n_cand_of(cfg);
    int32_t found = 0;
    *match_n = 0;
    for (int32_t c = 0; c < W; ++c) {
        match_end[c] = -1;
        copy_len[c] = 0;
        for (int32_t j = 0; j < cfg->k; ++j)
            copy_tokens[c * cfg->k + j] = -1;
    }
    for (int32_t j = 0; j < cfg->n_ngram && found == 0; ++j) {
        int32_t n = cfg->ngram_lens[j];
        if (L < n + 1)
            continue;
        /* ends from the most recent down */
        for (int32_t e = L - 2; e >= n - 1 && found < W; --e) {
            int same = 1;
            for (int32_t t = 0; t < n; ++t) {
                if (x[e - t] != x[L - 1 - t]) {
                    same = 0;
                    break;
                }
            }
            if (same) {
                match_end[found] = e;
                ++found;
            }
        }
        if (found > 0)
            *match_n = n;
    }
    for (int32_t c = 0; c < found; ++c) {
        int32_t start = match_end[c] + 1;
        int32_t len = L - start;
        if (len > cfg->k)
            len = cfg->k;
        copy_len[c] = len;
        for (int32_t j = 0; j < len; ++j)
            copy_tokens[c * cfg->k + j] = x[start + j];
    }
    return found;
}

/* Step 2 -- Sec. 3.2, Eq. 3: the probe is the linear score w^T H (the
 * sigmoid is monotone, so the decision uses the logit).  Each product of a
 * bf16 and a float is exact in long double (8 + 24 <= 64 significand bits);
 * the running sum carries a 64-bit significand, and the result is rounded
 * once to float. */
float oracle_probe(const uint16_t *h_bf16, const float *w, int32_t d, float bias)
{
    long double s = 0.0L;
    for (int32_t i = 0; i < d; ++i)
        s += (long double)bf16_to_float(h_bf16[i]) * (long double)w[i];
    s += (long double)bias;
    return (float)s;
}

/* Step 3 -- Sec. 3.3, Eq. 4 with the kappa-gram gate: copy iff the probe
 * clears the threshold AND a match of length >= kappa exists; otherwise the
 * neural draft is used as given. */
int32_t oracle_select(int32_t match_n, const int32_t *copy_len, const int32_t *copy_tokens,
                      float z, const int32_t *ntok, const int32_t *npar,
                      int32_t nn, int32_t R, const oracle_cfg *cfg,
                      int32_t *dtok, int32_t *dpar, int32_t *dn)
{
    int32_t use_copy = (match_n >= cfg->kappa) && (z >= cfg->theta);
    for (int32_t r = 0; r < R; ++r) {
        dtok[r] = -1;
        dpar[r] = -1;
    }
    if (use_copy) {
        /* the candidates one after another, each a chain from the anchor */
        int32_t node = 1;
        for (int32_t c = 0; c < n_cand_of(cfg); ++c) {
            for (int32_t i = 0; i < copy_len[c]; ++i) {
                dtok[node] = copy_tokens[c * cfg->k + i];
                dpar[node] = i == 0 ? 0 : node - 1;
                ++node;
            }
        }
        *dn = node;
    } else {
        if (nn < 1)
            nn = 1;
        if (nn > R)
            nn = R;
        *dn = nn;
        for (int32_t i = 1; i < nn; ++i) {
            dtok[i] = ntok[i];
            dpar[i] = npar ? npar[i] : i - 1;
        }
    }
    return use_copy;
}

/* Step 4a -- greedy verification at T = 0 (Sec. 2, App. A): the target's
 * choice at a position is the lowest index holding the largest value. */
int32_t oracle_argmax_row(const uint16_t *row_bf16, int32_t V)
{
    int32_t best = -1;
    float best_val = 0.0f;
    for (int32_t v = 0; v < V; ++v) {
        float f = bf16_to_float(row_bf16[v]);
        if (isnan(f))
            continue;
        if (best < 0 || f > best_val) {
            best = v;
            best_val = f;
        }
    }
    return best < 0 ? 0 : best;
}

/* Step 4a at T > 0 -- App. A measures SwitchSD at sampling temperatures
 * T > 0 with standard speculative sampling.  The target's distribution at a
 * drafted position is p = softmax(l / T).  It is realized with integer
 * weights w_j (see the header) so that every sum and every decision below is
 * exact integer arithmetic and does not depend on an order of summation. */
float oracle_sample_scale(float temperature)
{
    return (float)(1.4426950408889634 / (double)temperature);
}

/* 2^t for t in [-41, 0] as 2^k * P(f), k = rint(t), f = t - k in
 * [-1/2, 1/2] (exact), P(f) = sum_n (f ln 2)^n / n! up to n = 6, evaluated by
 * Horner's rule with one rounding per step (fused multiply-add).  The weight
 * is floor(2^40 * 2^k * P(f)); below t = -41 that is 0, and so is the weight
 * of NaN and -inf. */
uint64_t oracle_sample_weight(float l, float m, float c)
{
    const float t = (l - m) * c;
    if (!(t >= -41.0f))
        return 0u;
    const float k = rintf(t);
    const float f = t - k;
    float p = 0x1.430912p-13f;          /* ln2^6 / 6! */
    p = fmaf(p, f, 0x1.5d87fep-10f);    /* ln2^5 / 5! */
    p = fmaf(p, f, 0x1.3b2ab6p-7f);     /* ln2^4 / 4! */
    p = fmaf(p, f, 0x1.c6b08ep-5f);     /* ln2^3 / 3! */
    p = fmaf(p, f, 0x1.ebfbe0p-3f);     /* ln2^2 / 2! */
    p = fmaf(p, f, 0x1.62e430p-1f);     /* ln2 */
    p = fmaf(p, f, 1.0f);
    const float e = ldexpf(p, (int)k);  /* exact: a power-of-two scaling of a normal float */
    return (uint64_t)floor(ldexp((double)e, 40));
}

/* The weights of one row and their sum.  m is the largest non-NaN value.  A
 * row without a finite maximum (every value NaN, -inf, or +inf present) has
 * the one-hot weights 2^40 at its greedy choice (the lowest index of its
 * largest value) and 0 elsewhere. */
uint64_t oracle_row_weights(const uint16_t *row_bf16, int32_t V, float c, uint64_t *w)
{
    float m = 0.0f;
    int have = 0;
    for (int32_t v = 0; v < V; ++v) {
        const float f = bf16_to_float(row_bf16[v]);
        if (isnan(f))
            continue;
        if (!have || f > m)
            m = f;
        have = 1;
    }
    uint64_t Z = 0;
    if (!have || !isfinite(m)) {
        const int32_t g = oracle_argmax_row(row_bf16, V);
        for (int32_t v = 0; v < V; ++v)
            w[v] = v == g ? ((uint64_t)1 << 40) : 0u;
        return (uint64_t)1 << 40;
    }
    for (int32_t v = 0; v < V; ++v) {
        const float f = bf16_to_float(row_bf16[v]);
        w[v] = isnan(f) ? 0u : oracle_sample_weight(f, m, c);
        Z += w[v];
    }
    return Z;
}

/* Inverse CDF: the smallest j with w_0 + ... + w_j > floor(u * Z / 2^64). */
int32_t oracle_draw(const uint64_t *w, int32_t V, uint64_t Z, uint64_t u)
{
    const uint64_t target = (uint64_t)(((unsigned __int128)u * Z) >> 64);
    uint64_t prefix = 0;
    for (int32_t v = 0; v < V; ++v) {
        prefix += w[v];
        if (prefix > target)
            return v;
    }
    return V - 1; /* not reached: target < Z */
}

int32_t oracle_sample_row(const uint16_t *row_bf16, int32_t V, float c, uint64_t u)
{
    uint64_t *w = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(V > 0 ? V : 1));
    const uint64_t Z = oracle_row_weights(row_bf16, V, c, w);
    const int32_t y = oracle_draw(w, V, Z, u);
    free(w);
    return y;
}

/* 192-bit product of a 128-bit and a 64-bit unsigned integer, as its upper
 * 128 bits (hi) and lower 64 bits (lo). */
static void mul_128_64(unsigned __int128 a, uint64_t b, unsigned __int128 *hi, uint64_t *lo)
{
    const unsigned __int128 plo = (unsigned __int128)(uint64_t)a * b;
    const unsigned __int128 phi = (unsigned __int128)(uint64_t)(a >> 64) * b;
    *lo = (uint64_t)plo;
    *hi = phi + (plo >> 64);
}

/* Speculative sampling with the draft's own distribution q (Sec. 2,
 * Speculative Decoding; App. A at T > 0): the drafted token x is accepted with
 * probability min(1, p(x) / q(x)), p and q being the target's and the
 * draft's distributions at the parent position, both softmax(. / T) realized
 * with the integer weights above (P_j / Zp and Q_j / Zq).  With a 64-bit
 * uniform u the test is u / 2^64 < p(x) / q(x), i.e. in integers
 *   u * Q_x * Zp < 2^64 * P_x * Zq.
 * A token outside [0, V) has P_x = Q_x = 0 and is rejected. */
int32_t oracle_spec_accept(const uint16_t *p_row, const uint16_t *q_row, int32_t V, float c,
                           int32_t x, uint64_t u)
{
    uint64_t *P = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    uint64_t *Q = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    const uint64_t Zp = oracle_row_weights(p_row, V, c, P);
    const uint64_t Zq = oracle_row_weights(q_row, V, c, Q);
    const uint64_t Px = (x >= 0 && x < V) ? P[x] : 0u;
    const uint64_t Qx = (x >= 0 && x < V) ? Q[x] : 0u;
    free(P);
    free(Q);
    unsigned __int128 lhi;
    uint64_t llo;
    mul_128_64((unsigned __int128)u * Qx, Zp, &lhi, &llo);   /* u Q_x Zp */
    const unsigned __int128 rhi = (unsigned __int128)Px * Zq; /* 2^64 P_x Zq = (rhi, 0) */
    return lhi < rhi;
}

/* After a rejection the emitted token is drawn from the normalized residual
 * max(0, p - q) (Sec. 2; App. A), in integers
 *   R_j = max(0, P_j * Zq - Q_j * Zp),
 * by inverse CDF: the smallest j with R_0 + ... + R_j > floor(u * sum R / 2^64).
 * The residual has positive mass whenever a rejection is possible (p(x) < q(x)
 * for the drafted x); a row with none gives the draw from p instead. */
int32_t oracle_residual_row(const uint16_t *p_row, const uint16_t *q_row, int32_t V, float c,
                            uint64_t u)
{
    uint64_t *P = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    uint64_t *Q = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    const uint64_t Zp = oracle_row_weights(p_row, V, c, P);
    const uint64_t Zq = oracle_row_weights(q_row, V, c, Q);
    unsigned __int128 S = 0;
    for (int32_t j = 0; j < V; ++j) {
        const unsigned __int128 a = (unsigned __int128)P[j] * Zq;
        const unsigned __int128 b = (unsigned __int128)Q[j] * Zp;
        S += a > b ? a - b : 0;
    }
    int32_t y = V - 1;
    if (S == 0) {
        y = oracle_draw(P, V, Zp, u);
    } else {
        unsigned __int128 target;
        uint64_t lo;
        mul_128_64(S, u, &target, &lo);  /* floor(u S / 2^64) */
        unsigned __int128 prefix = 0;
        for (int32_t j = 0; j < V; ++j) {
            const unsigned __int128 a = (unsigned __int128)P[j] * Zq;
            const unsigned __int128 b = (unsigned __int128)Q[j] * Zp;
            prefix += a > b ? a - b : 0;
            if (prefix > target) {
                y = j;
                break;
            }
        }
    }
    free(P);
    free(Q);
    return y;
}

/* A chain drafted with distribution q (rows r of draft_logits: the draft
 * model's logits at node r, from which node r + 1 was drawn).  Rows are
 * tested in order; the first rejection at row r ends the step with the
 * residual draw there (accept_len = r); with no rejection the bonus is drawn
 * from p at the last drafted row.  amax[r] receives the token emitted at row
 * r (the drafted token when accepted, then the residual draw or the bonus)
 * and -1 at the rows after it. */
static void spec_chain(const uint16_t *logits, const uint16_t *qlogits, int64_t V, int32_t R,
                       const int32_t *dtok, int32_t dn, float c, const uint64_t *un,
                       const uint64_t *ua, int32_t *am, int32_t *accept_len,
                       int32_t *accept_node, int32_t *bonus, int32_t *out_tokens)
{
    int32_t a = dn - 1;
    for (int32_t r = 0; r + 1 < dn; ++r) {
        if (!oracle_spec_accept(logits + r * V, qlogits + r * V, (int32_t)V, c, dtok[r + 1],
                                ua[r])) {
            a = r;
            break;
        }
    }
    const int32_t y = a + 1 < dn ? oracle_residual_row(logits + a * V, qlogits + a * V,
                                                       (int32_t)V, c, un[a])
                                 : oracle_sample_row(logits + a * V, (int32_t)V, c, un[a]);
    for (int32_t r = 0; r < R; ++r) {
        am[r] = r < a ? dtok[r + 1] : (r == a ? y : -1);
        out_tokens[r] = r < a ? dtok[r + 1] : (r == a ? y : -1);
    }
    *accept_len = a;
    *accept_node = a;
    *bonus = y;
}

/* Step 4b -- Sec. 3.3 (select the longest validated continuation): a node is
 * accepted when its parent is accepted and its token equals the target's
 * choice at the parent.  The result is the deepest accepted node, the tokens
 * on its path and the target's own token after it (the bonus). */
void oracle_accept(const int32_t *dtok, const int32_t *dpar, int32_t dn,
                   const int32_t *amax, int32_t R,
                   int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                   int32_t *out_tokens)
{
    int32_t *accepted = (int32_t *)calloc((size_t)R, sizeof(int32_t));
    int32_t *depth = (int32_t *)calloc((size_t)R, sizeof(int32_t));
    accepted[0] = 1;
    depth[0] = 0;
    for (int32_t i = 1; i < dn; ++i) {
        int32_t p = dpar[i];
        if (p < 0 || p >= i)
            continue;
        if (accepted[p] && dtok[i] == amax[p]) {
            accepted[i] = 1;
            depth[i] = depth[p] + 1;
        }
    }
    int32_t best = 0;
    for (int32_t i = 1; i < dn; ++i)
        if (accepted[i] && depth[i] > depth[best])
            best = i;
    *accept_node = best;
    *accept_len = depth[best];
    *bonus = amax[best];
    for (int32_t r = 0; r < R; ++r)
        out_tokens[r] = -1;
    /* path tokens root -> best, root excluded, written back to front */
    int32_t node = best;
    for (int32_t pos = depth[best] - 1; pos >= 0; --pos) {
        out_tokens[pos] = dtok[node];
        node = dpar[node];
    }
    out_tokens[depth[best]] = *bonus;
    free(accepted);
    free(depth);
}

/* Sec. 3.3 (Parallel Verification with Block-Triangular Attention): a draft
 * token sees itself and the tokens on its path back to the anchor (and the
 * whole prefix, which is not part of this mask). */
void oracle_tree_mask(const int32_t *dpar, int32_t dn, int32_t R, int32_t words,
                      uint32_t *mask)
{
    for (int32_t i = 0; i < R; ++i)
        for (int32_t w = 0; w < words; ++w)
            mask[i * words + w] = 0;
    for (int32_t i = 0; i < dn; ++i) {
        int32_t node = i;
        for (;;) {
            mask[i * words + node / 32] |= 1u << (node % 32);
            if (node == 0)
                break;
            int32_t p = dpar[node];
            if (p < 0 || p >= node)
                break;
            node = p;
        }
    }
}

/* Sec. 3.3 (KV Cache Synchronization): when a copy draft is accepted the
 * draft model's cache lags behind; the accepted tokens are passed through the
 * draft model in its next forward pass.  This is the bookkeeping of that
 * rule plus the append of the step's tokens to the context. */
void oracle_commit(int32_t *x, int32_t *length, int32_t Lmax, const int32_t *out_tokens,
                   int32_t accept_len, int32_t use_copy, int32_t *draft_pos, int32_t *lag)
{
    int32_t L = *length;
    if (L < 0)
        L = 0;
    if (L > Lmax)
        L = Lmax;
    int32_t Lnew = L + accept_len + 1;
    if (Lnew > Lmax)
        Lnew = Lmax;
    for (int32_t i = 0; L + i < Lnew; ++i)
        x[L + i] = out_tokens[i];
    int32_t pos = use_copy ? *draft_pos : L + accept_len;
    if (pos < 0)
        pos = 0;
    if (pos > Lnew)
        pos = Lnew;
    *length = Lnew;
    *draft_pos = pos;
    *lag = Lnew - pos;
}

/* Sec. 3.2 (Problem Formulation): the training label of the copy-intent
 * probe.  A verbatim span of at least n tokens that appears earlier contains
 * windows of exactly n tokens that appear earlier at the same offsets, and
 * such a window is itself a span of n tokens, so the rule is: j is covered by
 * an n-token window that is not the first occurrence of its tokens. */
void oracle_copy_labels(const int32_t *x, int32_t L, int32_t Lmax, int32_t n,
                        uint8_t *labels)
{
    for (int32_t j = 0; j < Lmax; ++j)
        labels[j] = 0;
    if (n < 1 || L > Lmax)
        return;
    for (int32_t s = 1; s + n <= L; ++s) {
        int earlier = 0;
        for (int32_t s2 = 0; s2 < s && !earlier; ++s2) {
            int same = 1;
            for (int32_t t = 0; t < n; ++t) {
                if (x[s2 + t] != x[s + t]) {
                    same = 0;
                    break;
                }
            }
            earlier = same;
        }
        if (earlier)
            for (int32_t t = 0; t < n; ++t)
                labels[s + t] = 1;
    }
}

typedef struct {
    int32_t b0, b1;
    int32_t Lmax, d, R, V;
    const int32_t *tokens, *lengths;
    const uint16_t *hidden;
    const float *w;
    float bias;
    const int32_t *ntok, *npar, *nn;
    const uint16_t *logits;
    const oracle_cfg *cfg;
    int32_t *match_n, *match_end, *copy_len, *copy_tokens;
    float *z;
    int32_t *use_copy, *dtok, *dpar, *dn, *amax;
    int32_t *accept_len, *accept_node, *bonus, *out_tokens;
    float temperature;
    const uint64_t *uniforms;
    const uint16_t *qlogits;
    const uint64_t *accept_uniforms;
} step_job;

static void step_range(const step_job *j)
{
    const int64_t R = j->R, V = j->V, K = j->cfg->k, W = n_cand_of(j->cfg);
    for (int32_t b = j->b0; b < j->b1; ++b) {
        int32_t L = j->lengths[b];
        if (L < 0)
            L = 0;
        if (L > j->Lmax)
            L = j->Lmax;
        const int32_t *x = j->tokens + (int64_t)b * j->Lmax;
        oracle_match(x, L, j->cfg, &j->match_n[b], j->match_end + b * W, j->copy_len + b * W,
                     j->copy_tokens + b * W * K);
        j->z[b] = oracle_probe(j->hidden + (int64_t)b * j->d, j->w, j->d, j->bias);
        j->use_copy[b] = oracle_select(j->match_n[b], j->copy_len + b * W,
                                       j->copy_tokens + b * W * K,
                                       j->z[b], j->ntok + b * R,
                                       j->npar ? j->npar + b * R : NULL, j->nn[b], j->R,
                                       j->cfg, j->dtok + b * R, j->dpar + b * R, &j->dn[b]);
        int32_t *am = j->amax + b * R;
        const float c = j->temperature > 0.0f ? oracle_sample_scale(j->temperature) : 0.0f;
        if (j->temperature > 0.0f && j->qlogits && !j->use_copy[b]) {
            /* a neural chain with its distribution: speculative sampling */
            spec_chain(j->logits + (int64_t)b * R * V, j->qlogits + (int64_t)b * R * V, V,
                       j->R, j->dtok + b * R, j->dn[b], c, j->uniforms + b * R,
                       j->accept_uniforms + b * R, am, &j->accept_len[b],
                       &j->accept_node[b], &j->bonus[b], j->out_tokens + b * R);
            continue;
        }
        for (int32_t r = 0; r < j->R; ++r) {
            const uint16_t *row = j->logits + ((int64_t)b * R + r) * V;
            if (r >= j->dn[b])
                am[r] = -1;
            else if (j->temperature > 0.0f)
                am[r] = oracle_sample_row(row, j->V, c, j->uniforms[b * R + r]);
            else
                am[r] = oracle_argmax_row(row, j->V);
        }
        oracle_accept(j->dtok + b * R, j->dpar + b * R, j->dn[b], am, j->R,
                      &j->accept_len[b], &j->accept_node[b], &j->bonus[b],
                      j->out_tokens + b * R);
    }
}

static void *step_thread(void *arg)
{
    step_range((const step_job *)arg);
    return NULL;
}

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
                int32_t threads)
{
    if (B < 0 || Lmax < 1 || d < 0 || R < 1 || V < 1 || !cfg || cfg->k < 0 ||
        n_cand_of(cfg) * cfg->k + 1 > R)
        return -1;
    if (cfg->n_ngram < 1 || cfg->n_ngram > ORACLE_MAX_NGRAM)
        return -1;
    if (temperature > 0.0f && !uniforms)
        return -1;
    if (draft_logits && (!(temperature > 0.0f) || !accept_uniforms || npar))
        return -1;
    if (threads < 1)
        threads = 1;
    if (threads > B)
        threads = B > 0 ? B : 1;
    step_job base = {0, 0, Lmax, d, R, V, tokens, lengths, hidden, w, bias, ntok, npar, nn,
                     logits, cfg, match_n, match_end, copy_len, copy_tokens, z, use_copy,
                     dtok, dpar, dn, amax, accept_len, accept_node, bonus, out_tokens,
                     temperature, uniforms, draft_logits, accept_uniforms};
    if (threads == 1) {
        base.b0 = 0;
        base.b1 = B;
        step_range(&base);
        return 0;
    }
    step_job *jobs = (step_job *)malloc(sizeof(step_job) * (size_t)threads);
    pthread_t *tid = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)threads);
    for (int32_t t = 0; t < threads; ++t) {
        jobs[t] = base;
        jobs[t].b0 = (int32_t)((int64_t)B * t / threads);
        jobs[t].b1 = (int32_t)((int64_t)B * (t + 1) / threads);
        pthread_create(&tid[t], NULL, step_thread, &jobs[t]);
    }
    for (int32_t t = 0; t < threads; ++t)
        pthread_join(tid[t], NULL);
    free(jobs);
    free(tid);
    return 0;
}
