/*
 * CPU oracle for the beam-search decode step of FastSeq (arXiv 2106.04718).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or run this code.  It shares no code,
 * header, table or helper with the GPU library, and the GPU library never
 * calls it.
 *
 * It is deliberately plain: straight loops in the order of the definitions,
 * fp64 arithmetic for the attention, and no blocking, fusion or reordering.
 * OpenMP only spreads independent output rows over threads; each row is
 * computed by one thread in a fixed order, so the result does not depend on
 * the thread count.
 *
 *   oracle_cross_attn   encoder-decoder attention over a de-duplicated K/V
 *                       cache (Appendix B, Eq. 4), with a key-length mask.
 *   oracle_prefix_attn  self-attention with a shared prefix cache and a per-beam
 *                       generated-token cache (Appendix A, Eq. 2 and Eq. 3).
 *   oracle_cross_attn_replicated  the same over K/V replicated per beam (the
 *                       layout of Eq. 1), the form Eq. 4 replaces.
 *   oracle_ngram_block  no-repeat-n-gram blocking (Section 4.2, Algorithm 1)
 *                       written as its plain definition.
 *   oracle_ngram_banned the same bans as a sorted list of (row, token) pairs.
 *   oracle_beam_select  one beam-search selection step (Section 2.1) over
 *                       log-probabilities with the n-gram bans applied.
 *   oracle_cache_reorder the per-beam cache reorder that follows a selection
 *                       step (Section 2.2, cache maintenance; Section 4.1.1).
 *   oracle_ancestry_step the reorder-free form of that maintenance: a table of
 *                       which beam's cache row holds each generated token.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One (source, beam, head) row of Eq. 4: out = softmax(q K^T / sqrt(D)) V over
 * the first L rows of Kbh / Vbh ([S, D] each), in fp64.  L == 0 gives 0. */
static void attend_row(const double *qrow, const double *Kbh, const double *Vbh, int L, int D,
                       double *orow)
{
    if (L <= 0) {
        for (int d = 0; d < D; ++d) orow[d] = 0.0;
        return;
    }
    const double root_d = sqrt((double)D);
    double *w = (double *)malloc(sizeof(double) * (size_t)L);
    if (!w) abort();

    /* scores: s_j = (q . K_j) / sqrt(D) */
    for (int j = 0; j < L; ++j) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
            dot += qrow[d] * Kbh[(size_t)j * D + d];
        w[j] = dot / root_d;
    }
    /* softmax over the valid keys */
    double m = -INFINITY;
    for (int j = 0; j < L; ++j)
        if (w[j] > m) m = w[j];
    double Z = 0.0;
    for (int j = 0; j < L; ++j) {
        w[j] = exp(w[j] - m);
        Z += w[j];
    }
    /* weighted sum of the values */
    for (int d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int j = 0; j < L; ++j)
            acc += w[j] * Vbh[(size_t)j * D + d];
        orow[d] = acc / Z;
    }
    free(w);
}

static int clamp_len(int L, int S)
{
    return L < 0 ? 0 : (L > S ? S : L);
}

/*
 * Encoder-decoder attention with de-duplicated K/V (Appendix B, Eq. 4).
 *
 * Eq. 4 keeps one copy of the encoder keys and values per source,
 * Cache_K / Cache_V of shape [B, 1, N, D], and lets the B*M beam queries of
 * step t read it through an einsum; the result is the attention line of
 * Eq. 1, softmax(Q K^T / sqrt(d_k)) V, with K and V shared by the beams of a
 * source.  Written per head: every (source b, beam i, head h) is an
 * independent single-query attention over the keys of source b.
 *
 * Layouts (row-major, contiguous):
 *   q       [B, k, H, D]   query of beam i of source b (hypothesis b*k + i)
 *   K, V    [B, H, S, D]   one copy per source; rows j >= len are padding
 *   src_len [B]            valid keys of source b; clamped to [0, S]
 *   out     [B, k, H, D]
 *
 * Readings where the paper is silent: keys j >= src_len[b] take no weight
 * (they are never read); the scale 1/sqrt(D) multiplies the scores; the
 * softmax subtracts the row maximum, which leaves it unchanged
 * mathematically; an empty key set (len 0) gives a zero output row.
 *
 * Returns 0, or 1 for invalid sizes (nothing is written then).
 */
int oracle_cross_attn(const double *q, const double *K, const double *V,
                      const int32_t *src_len, double *out,
                      int B, int k, int H, int S, int D)
{
    if (B < 0 || k < 0 || H < 0 || S < 0 || D < 1)
        return 1;
    if (B == 0 || k == 0 || H == 0)
        return 0;
    if (!q || !K || !V || !src_len || !out)
        return 1;

    const long rows = (long)B * k * H;

#pragma omp parallel for schedule(dynamic, 4)
    for (long r = 0; r < rows; ++r) {
        /* r = (b*k + i)*H + h: source b, beam i, head h */
        const int h = (int)(r % H);
        const int b = (int)(r / ((long)H * k));
        const double *Kbh = K + ((size_t)b * H + h) * (size_t)S * D;
        const double *Vbh = V + ((size_t)b * H + h) * (size_t)S * D;
        attend_row(q + r * D, Kbh, Vbh, clamp_len(src_len[b], S), D, out + r * D);
    }
    return 0;
}

/*
 * The same attention over the conventional layout of Eq. 1, where the
 * encoder keys and values are replicated for every beam: K, V [B*k, H, S, D],
 * hypothesis b*k + i reading its own copy K[b*k + i] (with the length of its
 * source, src_len[b]).  With every copy of a source equal, Eq. 4 holds that
 * the result is that of oracle_cross_attn on one copy.
 * Returns 0, or 1 for invalid sizes (nothing is written then).
 */
int oracle_cross_attn_replicated(const double *q, const double *K, const double *V,
                                 const int32_t *src_len, double *out,
                                 int B, int k, int H, int S, int D)
{
    if (B < 0 || k < 0 || H < 0 || S < 0 || D < 1)
        return 1;
    if (B == 0 || k == 0 || H == 0)
        return 0;
    if (!q || !K || !V || !src_len || !out)
        return 1;

    const long rows = (long)B * k * H;

#pragma omp parallel for schedule(dynamic, 4)
    for (long r = 0; r < rows; ++r) {
        /* r = hyp*H + h with hyp = b*k + i */
        const int h = (int)(r % H);
        const long hyp = r / H;
        const int b = (int)(hyp / k);
        const double *Kbh = K + ((size_t)hyp * H + h) * (size_t)S * D;
        const double *Vbh = V + ((size_t)hyp * H + h) * (size_t)S * D;
        attend_row(q + r * D, Kbh, Vbh, clamp_len(src_len[b], S), D, out + r * D);
    }
    return 0;
}

/*
 * Self-attention over a split cache (Appendix A, Eq. 2 and Eq. 3).
 *
 * The prefix X of a sample (prompt or source, length N) is the same for all
 * its M beams, so its keys/values Cache_K', Cache_V' are kept once per
 * sample, [B, 1, N, D]; the keys/values of the t generated tokens, K_t and
 * V_t, differ per beam, [B*M, t, D].  Eq. 3 scores the query against both
 * parts, concatenates the scores, takes one softmax over the N + t entries,
 * splits the probabilities again and adds the two weighted sums.  Written
 * per head, with the steps in that order.
 *
 * Layouts (row-major, contiguous):
 *   q          [B, k, H, D]     query of beam i of sample b
 *   Kp, Vp     [B, H, N, D]     shared prefix; rows j >= prefix_len[b] are padding
 *   prefix_len [B]              valid prefix rows of sample b; clamped to [0, N]
 *   Kt, Vt     [B*k, H, T, D]   per-beam generated tokens; rows j >= t unused
 *   t          number of generated tokens of every beam (0 <= t <= T)
 *   out        [B, k, H, D]
 * Readings: the scale 1/sqrt(D) multiplies the scores; the softmax subtracts
 * the maximum; with no key at all (prefix_len 0 and t 0) the output is 0.
 * Returns 0, or 1 for invalid sizes (nothing is written then).
 */
int oracle_prefix_attn(const double *q, const double *Kp, const double *Vp,
                       const int32_t *prefix_len, const double *Kt, const double *Vt,
                       int t, double *out, int B, int k, int H, int N, int T, int D)
{
    if (B < 0 || k < 0 || H < 0 || N < 0 || T < 0 || D < 1 || t < 0 || t > T)
        return 1;
    if (B == 0 || k == 0 || H == 0)
        return 0;
    if (!q || !prefix_len || !out || (N > 0 && (!Kp || !Vp)) || (T > 0 && (!Kt || !Vt)))
        return 1;

    const double root_d = sqrt((double)D);
    const long rows = (long)B * k * H;

#pragma omp parallel for schedule(dynamic, 4)
    for (long r = 0; r < rows; ++r) {
        /* r = (b*k + i)*H + h: sample b, beam i, head h; hypothesis b*k + i */
        const int h = (int)(r % H);
        const long hyp = r / H;
        const int b = (int)(hyp / k);
        const double *qrow = q + r * D;
        double *orow = out + r * D;
        const double *Kpbh = Kp + ((size_t)b * H + h) * (size_t)N * D;
        const double *Vpbh = Vp + ((size_t)b * H + h) * (size_t)N * D;
        const double *Ktr = Kt + ((size_t)hyp * H + h) * (size_t)T * D;
        const double *Vtr = Vt + ((size_t)hyp * H + h) * (size_t)T * D;

        int P = prefix_len[b];
        if (P < 0) P = 0;
        if (P > N) P = N;
        const int n_all = P + t;
        if (n_all == 0) {
            for (int d = 0; d < D; ++d) orow[d] = 0.0;
            continue;
        }
        double *w = (double *)malloc(sizeof(double) * (size_t)n_all);
        if (!w) abort();

        /* attn_w0: scores against the shared prefix */
        for (int j = 0; j < P; ++j) {
            double dot = 0.0;
            for (int d = 0; d < D; ++d)
                dot += qrow[d] * Kpbh[(size_t)j * D + d];
            w[j] = dot;
        }
        /* attn_w1: scores against this beam's generated tokens */
        for (int j = 0; j < t; ++j) {
            double dot = 0.0;
            for (int d = 0; d < D; ++d)
                dot += qrow[d] * Ktr[(size_t)j * D + d];
            w[P + j] = dot;
        }
        /* attn_prob = softmax(concat(attn_w0, attn_w1) / sqrt(d)) */
        for (int j = 0; j < n_all; ++j)
            w[j] /= root_d;
        double m = w[0];
        for (int j = 1; j < n_all; ++j)
            if (w[j] > m) m = w[j];
        double Z = 0.0;
        for (int j = 0; j < n_all; ++j) {
            w[j] = exp(w[j] - m);
            Z += w[j];
        }
        for (int j = 0; j < n_all; ++j)
            w[j] /= Z;
        /* split; attn_t = attn_prob_0 . Cache_V' + attn_prob_1 . V_t */
        for (int d = 0; d < D; ++d) {
            double a0 = 0.0, a1 = 0.0;
            for (int j = 0; j < P; ++j)
                a0 += w[j] * Vpbh[(size_t)j * D + d];
            for (int j = 0; j < t; ++j)
                a1 += w[P + j] * Vtr[(size_t)j * D + d];
            orow[d] = a0 + a1;
        }
        free(w);
    }
    return 0;
}

/*
 * No-repeat-n-gram blocking (Section 4.2, Algorithm 1; Section 2.2).
 *
 * Definition: for hypothesis row r with generated tokens x_0 .. x_{t-1},
 * token v is banned iff the n-gram (x_{t-n+1}, .., x_{t-1}, v) already
 * occurs in the row, i.e. there is a window start j in [0, t-n] with
 * x_{j+c} == x_{t-n+1+c} for c = 0 .. n-2 and x_{j+n-1} == v.  A banned
 * token's logit is set to -inf (zero probability); every other logit is
 * left as it was.
 *
 * Readings: each window makes n-1 comparisons (the printed loop bound would
 * read one token past the row); the last window may overlap the trailing
 * n-1 tokens; token ids outside [0, V) are compared but never written;
 * t < n gives no window and changes nothing; n == 1 bans every token of
 * the row.
 *
 * Layouts: tokens [rows, ld] int32 (first t columns used), logits
 * [rows, V] fp32, modified in place.
 * Returns 0, or 1 for invalid arguments (nothing is written then).
 */
int oracle_ngram_block(const int32_t *tokens, int ld, int rows, int t, int n,
                       float *logits, int V)
{
    if (rows < 0 || t < 0 || n < 1 || V < 0 || ld < t)
        return 1;
    if (rows == 0 || t < n)
        return 0;
    if (!tokens || !logits)
        return 1;

#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        const int32_t *x = tokens + (size_t)r * ld;
        float *lg = logits + (size_t)r * V;
        const int suffix = t - n + 1; /* first of the trailing n-1 tokens */
        for (int j = 0; j <= t - n; ++j) {
            int same = 1;
            for (int c = 0; c < n - 1; ++c) {
                if (x[j + c] != x[suffix + c]) {
                    same = 0;
                    break;
                }
            }
            if (!same)
                continue;
            const int32_t v = x[j + n - 1];
            if (v >= 0 && v < V)
                lg[v] = -INFINITY;
        }
    }
    return 0;
}

/*
 * The bans of oracle_ngram_block as a list instead of writes: the pairs
 * (row r, token v), v in [0, V), such that some window j in [0, t-n] of row r
 * matches the row's last n-1 tokens and is followed by v.  Pairs are listed
 * by row, then by increasing v, each once; pairs[2p] = r, pairs[2p+1] = v.
 * At most max_pairs pairs are written; the return value is the number of
 * pairs (which may exceed max_pairs), or -1 for invalid arguments.
 */
static int cmp_i32(const void *a, const void *b)
{
    const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

long oracle_ngram_banned(const int32_t *tokens, int ld, int rows, int t, int n, int V,
                         int32_t *pairs, long max_pairs)
{
    if (rows < 0 || t < 0 || n < 1 || V < 0 || ld < t || max_pairs < 0)
        return -1;
    if (rows == 0 || t < n)
        return 0;
    if (!tokens || (max_pairs > 0 && !pairs))
        return -1;
    int32_t *found = (int32_t *)malloc(sizeof(int32_t) * (size_t)(t - n + 1));
    if (!found) abort();
    long count = 0;
    for (int r = 0; r < rows; ++r) {
        const int32_t *x = tokens + (size_t)r * ld;
        const int suffix = t - n + 1;
        int nf = 0;
        for (int j = 0; j <= t - n; ++j) {
            int same = 1;
            for (int c = 0; c < n - 1; ++c) {
                if (x[j + c] != x[suffix + c]) {
                    same = 0;
                    break;
                }
            }
            const int32_t v = x[j + n - 1];
            if (same && v >= 0 && v < V)
                found[nf++] = v;
        }
        qsort(found, (size_t)nf, sizeof(int32_t), cmp_i32);
        for (int f = 0; f < nf; ++f) {
            if (f > 0 && found[f] == found[f - 1])
                continue;
            if (count < max_pairs) {
                pairs[2 * count] = r;
                pairs[2 * count + 1] = found[f];
            }
            ++count;
        }
    }
    free(found);
    return count;
}

/*
 * Tokens banned for one hypothesis by no-repeat-n-gram blocking (Section
 * 4.2, Algorithm 1, with the readings of oracle_ngram_block): banned[v] = 1
 * for every v in [0, V) that follows an earlier occurrence of the row's last
 * n-1 tokens.  n == 0 bans nothing.
 */
static void row_bans(const int32_t *x, int t, int n, int V, unsigned char *banned)
{
    memset(banned, 0, (size_t)V);
    if (n < 1 || t < n)
        return;
    const int suffix = t - n + 1;
    for (int j = 0; j <= t - n; ++j) {
        int same = 1;
        for (int c = 0; c < n - 1; ++c) {
            if (x[j + c] != x[suffix + c]) {
                same = 0;
                break;
            }
        }
        const int32_t v = x[j + n - 1];
        if (same && v >= 0 && v < V)
            banned[v] = 1;
    }
}

/*
 * One beam-search selection step (Section 2.1: at every step beam search
 * keeps the best candidates of each source), over log-probabilities with
 * the no-repeat-n-gram bans of Algorithm 1 applied (Section 4.2).
 *
 * Source b has hypotheses r = b*k + i (i < k) with running log-probability
 * beam_scores[r].  With x = logits[r, :]:
 *   lse_r     = log(sum over every v of exp(x[v]))     (fp64, max subtracted)
 *   lp(r, v)  = x[v] - lse_r, or -inf if v is banned for row r
 *               (tokens[r, 0..t-1] with n; n == 0: no bans)
 *   cand(f)   = beam_scores[r] + lp(r, v),   f = i*V + v
 * Output for source b: the c largest candidates in descending order, equal
 * values in increasing f: out_scores[b, j] = cand(f), out_beam[b, j] = i,
 * out_token[b, j] = v.
 *
 * Readings: the normaliser covers every token, banned or not (a ban sets a
 * log-probability to -inf and does not renormalise the rest); a row whose
 * logits are all -inf has lp = -inf everywhere; -inf candidates are ordered
 * like any value (by f), so every c <= k*V is defined.  Logits are finite
 * or -inf.  The selection is the definition itself: c times, take the best
 * candidate not taken yet.
 *
 * Layouts: logits [B*k, V] fp32, beam_scores [B*k] fp32, tokens [B*k, ld]
 * int32 (first t columns; not read when n == 0), outputs [B, c].
 * Returns 0, or 1 for invalid arguments (nothing is written then).
 */
int oracle_beam_select(const float *logits, const float *beam_scores, const int32_t *tokens, int ld,
                       int t, int n, int B, int k, int V, int c,
                       double *out_scores, int32_t *out_beam, int32_t *out_token)
{
    if (B < 0 || k < 0 || V < 0 || c < 0 || n < 0 || (long long)c > (long long)k * V)
        return 1;
    if (n > 0 && (t < 0 || ld < t))
        return 1;
    if (B == 0 || c == 0)
        return 0;
    if (!logits || !beam_scores || (n > 0 && !tokens) || !out_scores || !out_beam || !out_token)
        return 1;
    const size_t nc = (size_t)k * V;
    int bad = 0;

#pragma omp parallel for schedule(dynamic)
    for (int b = 0; b < B; ++b) {
        double *cand = malloc(nc * sizeof(double));
        unsigned char *taken = calloc(nc, 1);
        unsigned char *banned = malloc((size_t)V > 0 ? (size_t)V : 1);
        if (!cand || !taken || !banned) {
#pragma omp atomic write
            bad = 1;
            free(cand);
            free(taken);
            free(banned);
            continue;
        }
        for (int i = 0; i < k; ++i) {
            const size_t r = (size_t)b * k + i;
            const float *x = logits + r * V;
            double mx = -INFINITY;
            for (int v = 0; v < V; ++v)
                if ((double)x[v] > mx)
                    mx = (double)x[v];
            double lse = -INFINITY;
            if (mx > -INFINITY) {
                double sum = 0.0;
                for (int v = 0; v < V; ++v)
                    sum += exp((double)x[v] - mx);
                lse = mx + log(sum);
            }
            row_bans(n > 0 ? tokens + r * ld : NULL, t, n, V, banned);
            for (int v = 0; v < V; ++v) {
                double lp = -INFINITY;
                if (lse > -INFINITY && !banned[v])
                    lp = (double)x[v] - lse;
                cand[(size_t)i * V + v] = (double)beam_scores[r] + lp;
            }
        }
        for (int j = 0; j < c; ++j) {
            size_t best = nc;
            for (size_t f = 0; f < nc; ++f) {
                if (taken[f])
                    continue;
                if (best == nc || cand[f] > cand[best])
                    best = f;
            }
            taken[best] = 1;
            out_scores[(size_t)b * c + j] = cand[best];
            out_beam[(size_t)b * c + j] = (int32_t)(best / (size_t)V);
            out_token[(size_t)b * c + j] = (int32_t)(best % (size_t)V);
        }
        free(cand);
        free(taken);
        free(banned);
    }
    return bad;
}

/*
 * Per-beam cache reorder after a selection step (Section 2.2, cache
 * maintenance; Section 4.1.1: with the cache split, only the per-beam part
 * Cache_K_t / Cache_V_t is reordered, the shared prefix never is).
 *
 * Beam search keeps k hypotheses per source; the new hypothesis j of source b
 * continues the old hypothesis parent[b*k + j] of the same source, so its
 * cache of generated tokens must hold what that parent's held.  For every
 * source b, beam j, head h and position tau < t:
 *     new[b*k + j, h, tau, :] = old[b*k + parent[b*k + j], h, tau, :]
 * Positions tau >= t (unused capacity) keep their bytes.  A parent outside
 * [0, k) leaves the row as it is (the hypothesis keeps its own history).
 *
 * The cache is raw bytes, esize bytes per element, [B*k, H, T, D] row-major;
 * it is rewritten in place from a copy of each source's old rows, so the
 * result does not depend on the order of the copies.
 * Returns 0, or 1 for invalid arguments (nothing is written then).
 */
int oracle_cache_reorder(unsigned char *cache, const int32_t *parent, int B, int k, int H, int T, int t, int D,
                         int esize)
{
    if (B < 0 || k < 1 || H < 0 || T < 0 || t < 0 || t > T || D < 0 || esize < 1)
        return 1;
    if ((long long)B * k * H * T * D == 0 || t == 0)
        return 0;
    if (!cache || !parent)
        return 1;
    const size_t row = (size_t)D * esize;              /* bytes of one (h, tau) vector */
    const size_t beam = (size_t)H * T * row;            /* bytes of one hypothesis */
    int bad = 0;

#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        unsigned char *src = cache + (size_t)b * k * beam;
        unsigned char *old = malloc((size_t)k * beam);
        if (!old) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        memcpy(old, src, (size_t)k * beam);
        for (int j = 0; j < k; ++j) {
            const int32_t pj = parent[(size_t)b * k + j];
            const int from = (pj >= 0 && pj < k) ? pj : j;
            for (int h = 0; h < H; ++h)
                for (int tau = 0; tau < t; ++tau)
                    memcpy(src + (size_t)j * beam + ((size_t)h * T + tau) * row,
                           old + (size_t)from * beam + ((size_t)h * T + tau) * row, row);
        }
        free(old);
    }
    return bad;
}

/*
 * Ancestry table of the generated-token cache: the same cache maintenance as
 * oracle_cache_reorder (Section 2.2; Section 4.1.1) without moving the rows.
 *
 * Each hypothesis writes the K/V of its tau-th generated token to its own
 * cache row, at position tau, and never moves it.  anc[r, tau] (tau <= the
 * step) is the beam, within r's source, whose row holds the tau-th token of
 * hypothesis r.  After a selection step at which each hypothesis holds t
 * tokens and the new hypothesis j of source b continues old beam
 * parent[b*k + j]:
 *     anc[b*k + j, tau] = old anc[b*k + parent[b*k + j], tau]   for tau < t
 *     anc[b*k + j, t]   = j          (the step's new token, in j's own row)
 * A parent outside [0, k) keeps the hypothesis' own history (as in
 * oracle_cache_reorder).  Reading row anc[r, tau] of r's source at position
 * tau then gives exactly what the physically reordered cache holds at
 * (r, tau).
 *
 * anc is [B*k, ld] int32 (ld > t), updated in place from a copy of each
 * source's old rows.  Returns 0, or 1 for invalid arguments.
 */
int oracle_ancestry_step(int32_t *anc, int ld, const int32_t *parent, int B, int k, int t)
{
    if (B < 0 || k < 1 || t < 0 || ld <= t)
        return 1;
    if (B == 0)
        return 0;
    if (!anc || !parent)
        return 1;
    int bad = 0;

#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        int32_t *src = anc + (size_t)b * k * ld;
        int32_t *old = malloc((size_t)k * ld * sizeof(int32_t));
        if (!old) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        memcpy(old, src, (size_t)k * ld * sizeof(int32_t));
        for (int j = 0; j < k; ++j) {
            const int32_t pj = parent[(size_t)b * k + j];
            const int from = (pj >= 0 && pj < k) ? pj : j;
            for (int tau = 0; tau < t; ++tau)
                src[(size_t)j * ld + tau] = old[(size_t)from * ld + tau];
            src[(size_t)j * ld + t] = j;
        }
        free(old);
    }
    return bad;
}

/* Number of OpenMP threads a parallel region of the oracle uses. */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the OpenMP thread count for later calls (n >= 1). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
