// Internal launch interface between the C ABI (capi.cpp) and the kernels.
// Arguments are already validated by the caller; these functions only size
// the grid, enqueue the kernels on `stream` and return hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fs {

// Records `msg` as the calling thread's fs_last_error() and returns `status`
// (the C ABI's error slot, shared by every entry point).
int set_error(int status, const char *msg);

// Keys per split-KV chunk of the cross-attention.  It depends only on the
// row size (D and element size), never on B, k or the lengths, so the
// reduction order -- and hence every output bit -- is the same whether a
// source is read by one beam or by k beams.
int cross_attn_chunk_keys(int D, int esize);

// How an attention call is decomposed (every path gives the same bits):
//   kSplit   one workgroup per (b, h, chunk), partial records merged by
//            trailing merger workgroups -- most parallel, pays a merge;
//   kWholeP  one workgroup per (b, h) of P*4 waves walking its chunks P at a
//            time -- no records, needs many (b, h) rows to fill the chip.
enum class AttnPath { kAuto = 0, kSplit, kWhole1, kWhole2, kWhole4 };

// The path for n_bh = B*H rows of at most jobs_max jobs (chunks, plus the
// generated tokens of the split cache): the size rule, unless a path was
// forced with set_attn_path_override.
AttnPath choose_attn_path(int n_bh, int jobs_max);

// Workgroup timelines of trace builds (trace.h): the buffer the attention
// kernels and the selection kernel write (8 words per workgroup, `cap`
// workgroups; null: none).  hipErrorNotSupported in other builds.
hipError_t set_attn_trace(unsigned long long *buf, unsigned int cap);
hipError_t set_select_trace(unsigned long long *buf, unsigned int cap);

// Process-wide overrides of the size rules, for tests and measurements
// (fs_set_tuning).  kAuto / 0 restore the rules; each returns the previous value.
AttnPath set_attn_path_override(AttnPath p);
int set_select_slices_override(int slices);

// Workspace size in 4-byte words: the per-tile partial records (plus one
// record per (b, h) for the generated-token segment when `split`), then one
// 64-bit counter per (b, h) for captured calls.
size_t cross_attn_workspace_floats(int B, int k, int H, int S, int D, int esize, bool split);

// The n-gram part of a fused decode step (the arguments of fs_ngram_block):
// its rows are scanned by extra workgroups of the attention launch.
struct NgramRows {
    const int32_t *tokens;
    int ld, rows, t, n;
    float *logits;
    int V;
};

// `epoch` in [1, 2^31) must differ from the epoch of every earlier call that
// used the same workspace: it tags the partial records, which are never
// cleared.  Epoch 0 (a call captured into a graph) tags them by the rows'
// counters in the workspace instead, which the kernels advance.  With `ngram` (rows > 0, t >= n) the launch also applies the
// n-gram bans.
// `path` is the decomposition choose_attn_path gave for the call.
hipError_t launch_cross_attn(const void *q, const void *K, const void *V,
                             const int32_t *src_len, void *out,
                             int B, int k, int H, int S, int D, bool bf16,
                             float *workspace, unsigned long long epoch, hipStream_t stream,
                             AttnPath path, const NgramRows *ngram = nullptr);

// Split-cache self-attention: shared prefix Kp/Vp [B,H,N,D] with
// prefix_len[B], per-beam generated tokens Kt/Vt [B*k,H,T,D] (rows < t).
// anc: [B*k, ld_anc] int32 ancestry table of the generated rows, or null
// (each hypothesis reads its own rows).
hipError_t launch_prefix_attn(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                              const void *Kt, const void *Vt, int T, int t, const int32_t *anc, int ld_anc,
                              void *out, int B, int k, int H, int N, int D, bool bf16, float *workspace,
                              unsigned long long epoch, hipStream_t stream, AttnPath path);

hipError_t launch_ngram_block(const int32_t *tokens, int ld_tokens, int rows, int t,
                              int n, float *logits, int V, hipStream_t stream);

// Beam selection: vocabulary slices per hypothesis row, the most candidates
// one source's ranking takes (k * slices * c) and the most record words it
// reads (k * slices * (2 + 2c)), and the workspace in 64-bit words (the
// records, then one counter per source).  Record words carry `epoch` (in [1,
// 2^31)) as their tag, or, with epoch 0 (a captured call), the source's
// counter with bit 31 set.
int beam_select_slices(int rows, int V, int k, int c);
int beam_select_max_candidates();
int beam_select_max_record_words();
size_t beam_select_workspace_words(int B, int k, int V, int c);
hipError_t launch_beam_select(const float *logits, const float *beam_scores, const int32_t *tokens, int ld,
                              int t, int n, float *out_scores, int32_t *out_beam, int32_t *out_token, int B,
                              int k, int V, int c, unsigned long long *workspace, unsigned long long epoch,
                              hipStream_t stream);

// Per-beam cache reorder: the chunk size (16 or 4 bytes) the kernel uses for
// these pointers and sizes, and the launch (K and, if not null, V).
int cache_reorder_chunk(const void *K, const void *V, int T, int t, int D, int esize);
hipError_t launch_cache_reorder(void *K, void *V, const int32_t *parent, int B, int k, int H, int T, int t, int D,
                                int esize, hipStream_t stream);
// Ancestry table step: columns < t from the parents, column t the own index.
hipError_t launch_ancestry_step(int32_t *anc, int ld, const int32_t *parent, int B, int k, int t,
                                hipStream_t stream);

}  // namespace fs
