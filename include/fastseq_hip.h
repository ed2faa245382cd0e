/*
 * fastseq_hip.h -- C ABI of the MI355X (gfx950) beam-search decode step.
 *
 * Two operations of FastSeq (arXiv 2106.04718) on one GPU:
 *
 *   fs_beam_cross_attn  encoder-decoder attention in which the k beam
 *                       queries of a source read that source's single,
 *                       de-duplicated K/V copy (Section 4.1.2; Appendix B,
 *                       Eq. 4).
 *   fs_ngram_block      no-repeat-n-gram blocking on the GPU (Section 4.2,
 *                       Algorithm 1): logits of tokens that would repeat an
 *                       earlier n-gram become -inf, in place.
 *   fs_beam_decode_step both of the above in one launch: the decode step's
 *                       cross-attention with its n-gram rows scanned by extra
 *                       workgroups of the same grid.
 *   fs_beam_prefix_attn self-attention over a split cache: the prefix shared
 *                       by a sample's beams is stored once (Section 4.1.1;
 *                       Appendix A, Eq. 2-3).
 *   fs_beam_select      one beam-search selection step (Section 2.1): the n-gram
 *                       bans, the log-softmax and each source's best
 *                       candidates in one pass over the logits.
 *   fs_cache_reorder    the per-beam cache reorder after a selection step
 *                       (Section 2.2, cache maintenance; Section 4.1.1), in
 *                       place.
 *   fs_beam_ancestry_step, fs_beam_prefix_attn_indirect
 *                       the same maintenance without moving rows: an ancestry
 *                       table of the generated tokens, and the split-cache
 *                       attention that reads its generated rows through it.
 *   fs_postproc_*       asynchronous post-processing (Section 4.3): a host
 *                       thread detokenises finished hypotheses while the GPU
 *                       generates the next batch.
 *
 * Conventions shared by every entry point
 *   - Pointers named "device" are HIP device memory; the caller owns every
 *     buffer.  The library never allocates, frees or synchronises in these
 *     calls; it only enqueues kernels on `stream` (a hipStream_t; NULL means
 *     the default stream) and returns.  A kernel fault surfaces at the
 *     caller's next synchronisation.
 *   - Arrays are row-major and contiguous unless a leading dimension is
 *     passed.
 *   - Argument errors are found on the host before any launch and leave all
 *     outputs untouched.  The return value is an fs_status_t; its detail is
 *     in fs_last_error().
 *   - Calls are re-entrant; calls on different streams may run concurrently
 *     as long as they do not share an output or workspace buffer.
 *   - Graph capture: every call may be captured into a HIP graph and
 *     replayed (FS_VALIDATE mode aside).  Calls whose workgroups exchange
 *     tagged records through the workspace (the attention's split-KV form
 *     for fewer than 128 (source, head) rows, and fs_beam_select) tag them,
 *     when captured, by a counter per row or source kept at the end of the
 *     workspace, which each replay advances on the device; eager calls tag
 *     them by a host epoch, and the two kinds of tag never coincide.  A
 *     workspace used by captured calls must keep serving calls of the same
 *     sizes while the graph is replayed (zero-fill it again before it serves
 *     other sizes under capture), and a graph's replays must not overlap
 *     other calls on the same workspace.
 *   - Debug mode: with the environment variable FS_VALIDATE=1 set when the
 *     library is first used (or after fs_set_tuning(FS_TUNE_VALIDATE, 1)),
 *     the attention calls copy src_len / prefix_len
 *     to the host (synchronising `stream`) and return FS_ERR_INVALID_ARG if
 *     a length lies outside [0, S] instead of clamping it; on a capturing
 *     stream, where that copy cannot run, they return FS_ERR_UNSUPPORTED.
 */
#ifndef FASTSEQ_HIP_H
#define FASTSEQ_HIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FS_ABI_VERSION 1

typedef enum {
    FS_OK = 0,
    FS_ERR_INVALID_ARG = 1,  /* bad pointer, size, alignment, aliasing or workspace */
    FS_ERR_UNSUPPORTED = 2,  /* valid but not implemented: D, k or dtype outside the set below,
                                or FS_VALIDATE mode under stream capture */
    FS_ERR_HIP = 3           /* a HIP runtime call or kernel launch failed */
} fs_status_t;

typedef enum {
    FS_F32 = 0,   /* IEEE binary32 */
    FS_BF16 = 1   /* bfloat16 (upper half of a binary32) */
} fs_dtype_t;

/* FS_ABI_VERSION of the built library. */
int fs_abi_version(void);

/* Static name of a status code ("FS_OK", ...); "unknown status" otherwise. */
const char *fs_status_string(int status);

/* Detail of the status returned by the calling thread's last call into the
 * library ("" if it returned FS_OK).  Owned by the library; valid until the
 * thread's next call. */
const char *fs_last_error(void);

/*
 * Workspace, in bytes, that fs_beam_cross_attn needs for these sizes
 * (per-tile softmax partials, fp32 values tagged with the call).  Zero-fill
 * it before its first use.  0 for empty problems; (size_t)-1 for
 * invalid or unsupported sizes.  The size depends on every argument, so
 * query it again whenever one changes.
 */
size_t fs_beam_cross_attn_workspace_bytes(int B, int k, int H, int S, int D, int dtype);

/*
 * Encoder-decoder attention over a de-duplicated K/V cache (Section 4.1.2;
 * Appendix B, Eq. 4).
 *
 * For every source b, beam i < k and head h, with L = clamp(src_len[b], 0, S):
 *     s_j          = (q[b,i,h,:] . K[b,h,j,:]) / sqrt(D)        for j < L
 *     out[b,i,h,:] = sum_j softmax(s)_j * V[b,h,j,:]
 * and out[b,i,h,:] = 0 when L == 0.  Rows j >= L of K and V are never read
 * (they may hold anything, NaN included).  The k beams of source b are the
 * hypotheses b*k .. b*k+k-1 of the flattened B*k batch; all of them read the
 * one copy K[b], V[b], which is never replicated per beam.
 *
 * Arguments (all device pointers except the sizes):
 *   q        [B, k, H, D]  dtype    queries of step t
 *   K, V     [B, H, S, D]  dtype    encoder keys/values, one copy per source
 *   src_len  [B]           int32    valid keys per source (right padding)
 *   out      [B, k, H, D]  dtype    result, rounded to nearest-even from fp32
 *   workspace, workspace_bytes      scratch of at least
 *            fs_beam_cross_attn_workspace_bytes(B, k, H, S, D, dtype)
 *            bytes (per-tile partials, then a counter per (source, head)
 *            row for captured calls).  It must be zero-filled once
 *            before its first use and not written by anything else after
 *            that: each call marks the words it writes with a tag of its
 *            own, and an all-zero or earlier-tagged word is never taken as
 *            this call's (an eager call's tag repeats only after 2^31 calls
 *            in one process, a captured call's after 2^31 replays).  Any
 *            size-compatible call may reuse it (also of
 *            fs_beam_prefix_attn).  Calls that share a workspace must not
 *            run concurrently.
 *   stream   hipStream_t (NULL = default stream)
 * Supported: dtype FS_F32 or FS_BF16, D in {16, 32, 64, 128}, 1 <= k <= 8,
 * B, H, S >= 0 with B*k*H below 2^31, a launch grid of about
 * B*H*S*D*esize/8192 workgroups (esize = 2 or 4 bytes) below 2^31, and one
 * (source, head) block of S*D*esize bytes below 2 GiB (0x7ff00000 bytes;
 * FS_ERR_UNSUPPORTED above).
 * Arithmetic: products and sums in fp32; the result does not depend on k,
 * B or the beam's position (bitwise), only on (L, S, D, dtype) and the data.
 * Errors: FS_ERR_INVALID_ARG for a null pointer with non-empty sizes,
 * negative sizes, a pointer of q/K/V/out/workspace not 16-byte aligned, a
 * workspace that is too small, or out or the workspace overlapping another
 * argument; sizes too large for one launch;
 * FS_ERR_UNSUPPORTED for D, k or dtype outside the set above; FS_ERR_HIP
 * for a failed launch.  B == 0, k == 0 or H == 0 returns FS_OK with no launch.
 */
int fs_beam_cross_attn(const void *q, const void *K, const void *V,
                       const int32_t *src_len, void *out,
                       int B, int k, int H, int S, int D, int dtype,
                       void *workspace, size_t workspace_bytes,
                       void *stream);

/*
 * Workspace, in bytes, that fs_beam_prefix_attn needs for these sizes (the
 * partials of fs_beam_cross_attn plus one per-beam record per source and
 * head for the generated tokens).  Zero-fill it before its first use.  0 for
 * empty problems; (size_t)-1 for
 * invalid or unsupported sizes.
 */
size_t fs_beam_prefix_attn_workspace_bytes(int B, int k, int H, int N, int T, int D, int dtype);

/*
 * Self-attention over a split cache (Section 4.1.1; Appendix A, Eq. 2 and
 * Eq. 3): the keys/values of the prefix (prompt) are stored once per sample
 * and shared by its k beams; those of the t generated tokens are stored per
 * beam.  One softmax covers both parts.
 *
 * For every sample b, beam i < k (hypothesis r = b*k + i) and head h, with
 * P = clamp(prefix_len[b], 0, N):
 *     s = concat((q . Kp[b,h,j,:])_{j<P}, (q . Kt[r,h,j,:])_{j<t}) / sqrt(D)
 *     out[b,i,h,:] = sum_{j<P} p_j Vp[b,h,j,:] + sum_{j<t} p_{P+j} Vt[r,h,j,:]
 * with p = softmax(s), and out = 0 when P + t == 0.  Rows j >= P of Kp/Vp and
 * rows j >= t of Kt/Vt are never read.
 *
 * Arguments (device pointers except the sizes):
 *   q          [B, k, H, D]     dtype  query of step t
 *   Kp, Vp     [B, H, N, D]     dtype  shared prefix, one copy per sample
 *   prefix_len [B]              int32  valid prefix rows per sample
 *   Kt, Vt     [B*k, H, T, D]   dtype  per-beam generated tokens; T is the
 *                                      capacity, rows 0..t-1 are used
 *   out        [B, k, H, D]     dtype
 *   workspace, workspace_bytes  at least fs_beam_prefix_attn_workspace_bytes
 *                               bytes, zero-filled before its first use
 *                               (the rules of fs_beam_cross_attn's workspace)
 * Supported sizes, dtypes, arithmetic, determinism and errors are those of
 * fs_beam_cross_attn (with N in the role of S); in addition t > T or a
 * negative T or t is FS_ERR_INVALID_ARG, and a (hypothesis, head) block of
 * T*D*esize bytes above 0x7ff00000 is FS_ERR_UNSUPPORTED.  The result bits do not depend on k,
 * B or the beam's position, nor on whether the prefix is shared or passed
 * replicated per beam.
 */
int fs_beam_prefix_attn(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                        const void *Kt, const void *Vt, int T, int t, void *out,
                        int B, int k, int H, int N, int D, int dtype,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * No-repeat-n-gram blocking (Section 4.2, Algorithm 1; Section 2.2).
 *
 * For every row r < rows with history x = tokens[r, 0..t-1]: if some window
 * start j in [0, t-n] has x[j..j+n-2] == x[t-n+1..t-1] (the last n-1
 * tokens), then logits[r, x[j+n-1]] = -inf.  Each window makes n-1
 * comparisons; windows may overlap the last n-1 tokens.  Ids outside [0, V)
 * take part in comparisons but are never written.  Every other logit keeps
 * its bits.  Several windows banning one id write the same value.
 *
 * Arguments:
 *   tokens     [rows, ld_tokens] int32, device; columns 0..t-1 are read
 *   rows, t    hypotheses (B*k) and generated length; ld_tokens >= t
 *   n          n-gram size, >= 1 (n == 1 bans every token of the row)
 *   logits     [rows, V] fp32, device; modified in place
 *   stream     hipStream_t (NULL = default stream)
 * Errors: FS_ERR_INVALID_ARG for n < 1, negative sizes, ld_tokens < t,
 * null pointers with non-empty sizes, or logits overlapping tokens;
 * FS_ERR_HIP for a failed launch.  rows == 0 or t < n returns FS_OK with no
 * launch.
 */
int fs_ngram_block(const int32_t *tokens, int ld_tokens, int rows, int t, int n,
                   float *logits, int V, void *stream);

/*
 * One decode step of beam search in one launch: fs_beam_cross_attn followed
 * by fs_ngram_block on the step's hypotheses (Appendix B, Eq. 4; Section 4.2,
 * Algorithm 1).  The B*k rows of the n-gram scan are taken by extra
 * workgroups at the head of the attention grid, so the scan runs under the
 * attention's K/V stream instead of after it.  The results are bit for bit
 * those of the two calls:
 *     fs_beam_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype,
 *                        workspace, workspace_bytes, stream);
 *     fs_ngram_block(tokens, ld_tokens, B*k, t, n, logits, vocab, stream);
 * Arguments are those of the two calls (vocab is fs_ngram_block's V); the
 * workspace is fs_beam_cross_attn's.  Besides the errors of both calls,
 * FS_ERR_INVALID_ARG when logits overlap q, K, V, out, src_len or the
 * workspace, or tokens overlap out or the workspace.  When one half is
 * empty (B, k or H == 0; t < n or vocab == 0) only the other runs.
 */
int fs_beam_decode_step(const void *q, const void *K, const void *V, const int32_t *src_len, void *out,
                        int B, int k, int H, int S, int D, int dtype,
                        const int32_t *tokens, int ld_tokens, int t, int n, float *logits, int vocab,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * fs_beam_decode_step for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same step with no workspace argument.  The split-KV
 * decomposition (fewer than 128 (source, head) rows) keeps its partial
 * records in an array of FS_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends; the other decompositions use
 * no scratch.  The call allocates nothing and frees nothing; its first use
 * on a GPU enqueues a clear of that GPU's array on `stream`.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, other threads) race and must not be issued.
 * Arguments, results (bit for bit) and errors are those of
 * fs_beam_decode_step without the workspace; in addition
 * FS_ERR_UNSUPPORTED when the split-KV records of these sizes exceed
 * FS_NOALLOC_SCRATCH_BYTES (see fs_beam_cross_attn_workspace_bytes).
 */
#define FS_NOALLOC_SCRATCH_BYTES (8u << 20)
int fs_beam_decode_step_noalloc(const void *q, const void *K, const void *V, const int32_t *src_len, void *out,
                                int B, int k, int H, int S, int D, int dtype,
                                const int32_t *tokens, int ld_tokens, int t, int n, float *logits, int vocab,
                                void *stream);

/*
 * Tuning controls, for tests and measurements: they replace a size rule of
 * the library for every later call in the process (every thread).  Results
 * do not depend on them except where a call's documentation says so (the
 * slice count of fs_beam_select).  Returns the previous value, or -1 for an
 * unknown knob or value (nothing changes then).
 *   FS_TUNE_ATTN_PATH      decomposition of the attention calls:
 *                          FS_ATTN_PATH_AUTO (the size rule), _SPLIT (one
 *                          workgroup per chunk of 256 keys at D = 64 bf16, with
 *                          partial records), _WHOLE1/_WHOLE2/_WHOLE4 (one
 *                          workgroup of 4/8/16 waves per (source, head)).
 *                          Every decomposition gives the same bits.
 *   FS_TUNE_SELECT_SLICES  vocabulary slices per row of fs_beam_select
 *                          (0: the size rule), within that call's limits.
 *   FS_TUNE_VALIDATE       debug mode on (1) or off (0); it starts as the
 *                          environment variable FS_VALIDATE sets it.
 */
enum {
    FS_TUNE_ATTN_PATH = 1,
    FS_TUNE_SELECT_SLICES = 2,
    FS_TUNE_VALIDATE = 3
};
enum {
    FS_ATTN_PATH_AUTO = 0,
    FS_ATTN_PATH_SPLIT = 1,
    FS_ATTN_PATH_WHOLE1 = 2,
    FS_ATTN_PATH_WHOLE2 = 3,
    FS_ATTN_PATH_WHOLE4 = 4
};
int fs_set_tuning(int knob, int value);

/*
 * Workgroup timelines, for measurement (not a method of the paper).  A
 * library built with tracing (build.py: build(trace=True), which compiles
 * every kernel with FS_TRACE=1) makes the attention kernels that take one
 * workgroup per (source, head) row and the selection kernel write, for
 * every workgroup g of each later launch, 8 64-bit words at buffer[8 g ..]
 * (clock stamps of the 100 MHz s_memrealtime counter, the hardware ids of
 * the compute unit, and counts; trace.h and the kernels list each word).
 * Workgroups past bytes / 64 write nothing.  NULL stops tracing.  The
 * buffer is device memory the caller owns; launches that overlap write
 * the same words.
 * Errors: FS_ERR_UNSUPPORTED in a library built without tracing (every
 * normal build: its kernels contain no tracing code); FS_ERR_INVALID_ARG
 * for a null buffer with bytes > 0 or one not 8-byte aligned; FS_ERR_HIP if
 * the device symbol cannot be set.
 */
int fs_trace_set(void *buffer, size_t bytes);

/*
 * Workspace, in bytes, that fs_beam_select needs for these sizes (per
 * (hypothesis, vocabulary slice) partial records, then a counter per source
 * for captured calls).  Zero-fill it before its
 * first use; the reuse rules are those of fs_beam_cross_attn's workspace.
 * 0 for empty problems; (size_t)-1 for invalid or unsupported sizes.
 */
size_t fs_beam_select_workspace_bytes(int B, int k, int V, int c);

/*
 * One beam-search selection step (Section 2.1: at every step beam search
 * keeps the best candidates of each source) with the no-repeat-n-gram bans
 * of Section 4.2, Algorithm 1, in one pass over the logits.
 *
 * Source b has hypotheses r = b*k + i (i < k) with running log-probabilities
 * beam_scores[r].  With x = logits[r, :]:
 *     lse_r      = log(sum over every v of exp(x[v]))
 *     cand(i*V+v) = beam_scores[r] + x[v] - lse_r, or -inf if v is banned for
 *                   row r (the rule of fs_ngram_block on tokens[r, 0..t-1])
 * and out_*[b, 0..c-1] are the c largest candidates of source b, best first,
 * equal values in increasing flat index i*V + v: out_scores the value,
 * out_beam the beam i, out_token the token v.  The normaliser covers every
 * token, banned or not (a ban sets a log-probability to -inf and does not
 * renormalise the rest).  A row whose logits are all -inf has -inf
 * candidates; -inf candidates are ordered by flat index like any value.
 *
 * Arguments (device pointers except the sizes):
 *   logits       [B*k, V] fp32, finite or -inf; read once, never written
 *   beam_scores  [B*k]    fp32
 *   tokens       [B*k, ld_tokens] int32, columns 0..t-1; not read if n == 0
 *   t, n         history length and n-gram size; n == 0 bans nothing
 *   out_scores   [B, c] fp32;  out_beam, out_token [B, c] int32
 *   workspace, workspace_bytes  at least fs_beam_select_workspace_bytes
 *                bytes, zero-filled before its first use
 *   stream       hipStream_t (NULL = default stream)
 * Supported: 1 <= c <= 16 and c <= k*V, 1 <= k <= 16, V >= 1, and for one
 * source at most 1024 candidates in the final ranking (k * c * slices, where
 * a row is cut into slices of at most 16381 logits) and 2048 partial-record
 * words (k * slices * (2 + 2c)); the slice count is reduced to fit these
 * when it can be, so only a vocabulary above 16381 * (1024 / (k * c))
 * logits can exceed them.  The slice count follows from the sizes;
 * fs_set_tuning(FS_TUNE_SELECT_SLICES, n) sets it within the same limits.
 * Arithmetic: fp32 (the normaliser from per-slice maxima and sums of exp);
 * the order and the bits of the result depend on the data, the slice count
 * and the address of logits modulo 16 bytes, never on run or launch.
 * Errors: FS_ERR_INVALID_ARG for null pointers with non-empty sizes, negative
 * sizes, n < 0, ld_tokens < t with n > 0, c > k*V, pointers not 4-byte
 * aligned, a workspace that is too small, or an output overlapping an input
 * or another output; FS_ERR_UNSUPPORTED for c, k or the candidate count
 * outside the set above; FS_ERR_HIP for a failed launch.  B == 0 returns
 * FS_OK with no launch.  If a partial record is not seen within about 10 ms
 * (which does not happen in a working launch), the source's outputs are NaN
 * and -1.
 */
int fs_beam_select(const float *logits, const float *beam_scores, const int32_t *tokens, int ld_tokens,
                   int t, int n, float *out_scores, int32_t *out_beam, int32_t *out_token,
                   int B, int k, int V, int c, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Per-beam cache reorder after a selection step (Section 2.2: beam search
 * reorders the cached keys and values of the kept beams at every step;
 * Section 4.1.1: with the cache split, only the per-beam part Cache_K_t /
 * Cache_V_t is reordered, the shared prefix and the encoder cache never are).
 *
 * The new hypothesis j of source b continues the old hypothesis
 * parent[b*k + j] of the same source.  In place, for every head h and
 * position tau < t:
 *     K[b*k + j, h, tau, :] = old K[b*k + parent[b*k + j], h, tau, :]
 * and the same for V.  Positions tau >= t keep their bytes; a hypothesis whose
 * parent is itself, or outside [0, k), keeps its rows (they are neither read
 * nor written).  Byte copies: the result is exact for any dtype.
 *
 * Arguments (device pointers except the sizes):
 *   K, V     [B*k, H, T, D] of dtype; V may be NULL (then only K moves)
 *   parent   [B*k] int32, the old beam (within the source) each new beam
 *            continues, e.g. the beams a selection step kept
 *   T, t     capacity and used positions of the cache (0 <= t <= T)
 *   dtype    FS_F32 or FS_BF16
 *   stream   hipStream_t (NULL = default stream)
 * Supported: 1 <= k <= 16 and D*esize a multiple of 4 bytes.  16-byte moves
 * when the pointers are 16-byte aligned and T*D*esize and t*D*esize are
 * multiples of 16; 4-byte moves otherwise.
 * Errors: FS_ERR_INVALID_ARG for negative sizes, t > T, null K or parent,
 * pointers not 4-byte aligned, K overlapping V, or parent overlapping the
 * cache; FS_ERR_UNSUPPORTED for k, dtype or D outside the set above or a
 * cache too large for one launch; FS_ERR_HIP for a failed launch.  B, H, D
 * or t == 0 returns FS_OK with no launch.
 */
int fs_cache_reorder(void *K, void *V, const int32_t *parent, int B, int k, int H, int T, int t, int D, int dtype,
                     void *stream);

/*
 * Ancestry table of the generated-token cache: the per-beam maintenance of
 * fs_cache_reorder (Section 2.2; Section 4.1.1) without moving any row.
 * Each hypothesis writes the K/V of its tau-th generated token to its own
 * row at position tau and never moves it; anc[r, tau] is the beam, within
 * r's source, whose row holds the tau-th token of hypothesis r.  After a
 * selection step at which every hypothesis holds t tokens, and before the
 * step's new token is written:
 *     anc[b*k + j, tau] = old anc[b*k + parent[b*k + j], tau]   tau < t
 *     anc[b*k + j, t]   = j
 * in place.  Columns past t keep their values; a parent outside [0, k)
 * keeps the hypothesis' own history.  Start from any table with t = 0.
 *
 * Arguments (device pointers except the sizes):
 *   anc      [B*k, ld_anc] int32, updated in place (t < ld_anc)
 *   parent   [B*k] int32, the old beam each new hypothesis continues
 *   stream   hipStream_t (NULL = default stream)
 * Supported: 1 <= k <= 16.
 * Errors: FS_ERR_INVALID_ARG for negative sizes, t >= ld_anc, null or
 * misaligned pointers, or parent overlapping anc; FS_ERR_UNSUPPORTED for k
 * or a table too large; FS_ERR_HIP for a failed launch.  B == 0 returns
 * FS_OK with no launch.
 */
int fs_beam_ancestry_step(int32_t *anc, int ld_anc, const int32_t *parent, int B, int k, int t, void *stream);

/*
 * fs_beam_prefix_attn with the generated rows read through an ancestry
 * table (fs_beam_ancestry_step): for hypothesis r = b*k + i, generated row
 * tau (tau < t) is row tau of the block of hypothesis b*k + anc[r, tau] of
 * Kt/Vt; an entry outside [0, k) reads r's own block.  Everything else --
 * arguments, layouts, the prefix part, errors -- is that of
 * fs_beam_prefix_attn; with anc[r, tau] = i for all tau it returns the same
 * bits.  The rows of one source's k beams are read through one buffer
 * range, so k*H*T*D*esize must stay below 2 GiB.
 *   anc      [B*k, ld_anc] int32 (ld_anc >= t); not read when t == 0
 * Additional errors: FS_ERR_INVALID_ARG for a null or misaligned anc with
 * t > 0, ld_anc < t, or out overlapping anc; FS_ERR_UNSUPPORTED for the
 * 2 GiB limit.
 */
int fs_beam_prefix_attn_indirect(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                                 const void *Kt, const void *Vt, const int32_t *anc, int ld_anc, int T, int t,
                                 void *out, int B, int k, int H, int N, int D, int dtype, void *workspace,
                                 size_t workspace_bytes, void *stream);

/*
 * Asynchronous post-processing of finished hypotheses (Section 4.3): a host
 * thread detokenises and writes out batch i while the GPU generates batch
 * i + 1.  A handle owns `slots` staging buffers of pinned host memory of
 * max_rows x max_len ids each (hipHostMalloc), one event per slot and the
 * worker thread; it is the only part of the library that allocates, and it
 * does so in fs_postproc_create only.
 *
 * Detokenisation is byte-level: token v is the UTF-8 text
 * vocab[offsets[v] .. offsets[v+1]) over an alphabet of one symbol per byte
 * -- a printable byte (0x21-0x7E, 0xA1-0xAC, 0xAE-0xFF) stands for itself,
 * the other bytes in increasing order are the code points 0x100, 0x101, ...
 * -- and the output bytes are recovered symbol by symbol (other characters
 * are dropped).  Each row becomes one line: the bytes of its ids up to its
 * first `eos` id (or its length), then '\n'; ids outside [0, V) are skipped.
 * Batches are written in submission order, rows in order.
 *
 *   fs_postproc_create   copies the vocabulary, opens `path` for writing (NULL:
 *                        keep the bytes in memory), allocates the staging and
 *                        starts the worker.  *out receives the handle.
 *   fs_postproc_submit   tokens [rows, ld] int32 in device memory (columns
 *                        0..t-1): enqueues their copy into the next staging
 *                        buffer on `stream` (after the work already on it)
 *                        and an event, hands the batch to the worker and
 *                        returns; it waits only while that buffer's previous
 *                        batch is not written yet.  One submitting thread.
 *   fs_postproc_flush    waits until every submitted batch is written (and
 *                        the file flushed); reports the first worker error.
 *   fs_postproc_output   between a flush and the next submit: the bytes kept
 *                        in memory -- copies at most cap of them into buf and
 *                        returns their total size.
 *   fs_postproc_busy_seconds  host time the worker has spent detokenising and
 *                        writing (not waiting).
 *   fs_postproc_destroy  finishes the submitted batches, stops the worker and
 *                        frees the handle.
 * Errors: FS_ERR_INVALID_ARG for null pointers, sizes below 1 or above the
 * staging, decreasing offsets or an unopenable path; FS_ERR_UNSUPPORTED for
 * staging above 2^31 ids; FS_ERR_HIP for a failed allocation, copy or event.
 */
typedef struct fs_postproc fs_postproc;
int fs_postproc_create(fs_postproc **out, const char *vocab, const int64_t *offsets, int V, int eos, int max_rows,
                       int max_len, int slots, const char *path);
int fs_postproc_submit(fs_postproc *pp, const int32_t *tokens, int ld, int rows, int t, void *stream);
int fs_postproc_flush(fs_postproc *pp);
size_t fs_postproc_output(fs_postproc *pp, char *buf, size_t cap);
double fs_postproc_busy_seconds(fs_postproc *pp);
void fs_postproc_destroy(fs_postproc *pp);

#ifdef __cplusplus
}
#endif

#endif /* FASTSEQ_HIP_H */
