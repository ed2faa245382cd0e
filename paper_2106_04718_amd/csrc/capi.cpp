// C ABI of the decode-step library: argument validation, status codes and
// dispatch to the kernels.  Every check here runs on the host before any HIP
// call, so invalid arguments never reach the GPU and leave outputs untouched.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "fastseq_hip.h"
#include "launch.h"

namespace {

thread_local std::string g_last_error;

int fail(int status, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

}  // namespace

int fs::set_error(int status, const char *msg) {
    g_last_error = msg;
    return status;
}

namespace {

int hip_fail(hipError_t e, const char *what) {
    return fail(FS_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Do the byte ranges [a, a+na) and [b, b+nb) intersect?
bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    if (na == 0 || nb == 0) return false;
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + nb && pb < pa + na;
}

// Debug mode: FS_VALIDATE=1 in the environment when the library is first
// used, or fs_set_tuning(FS_TUNE_VALIDATE, 1).
std::atomic<int> g_validate{-1};   // -1: not read from the environment yet

bool validate_mode() {
    int v = g_validate.load(std::memory_order_relaxed);
    if (v < 0) {
        const char *e = std::getenv("FS_VALIDATE");
        int expected = -1;
        g_validate.compare_exchange_strong(expected, (e && e[0] == '1') ? 1 : 0, std::memory_order_relaxed);
        v = g_validate.load(std::memory_order_relaxed);
    }
    return v == 1;
}

// Epochs tag the partial records in the workspace: every call gets a fresh
// epoch in [1, 2^31), so a workspace zero-filled once never needs clearing
// again (a zero word, or one left by an earlier call, never carries this
// call's tag).  Tags with bit 31 set belong to captured calls (below).
std::atomic<unsigned long long> g_epoch{0};

unsigned long long next_epoch() {
    return g_epoch.fetch_add(1, std::memory_order_relaxed) % 0x7fffffffull + 1;
}

bool supported_d(int D) { return D == 16 || D == 32 || D == 64 || D == 128; }

// Largest (source, head) block of K or V, in bytes: the kernels address one
// block through a 32-bit buffer range.
constexpr long long kMaxBlockBytes = 0x7ff00000LL;

static_assert((int)fs::AttnPath::kSplit == FS_ATTN_PATH_SPLIT && (int)fs::AttnPath::kWhole1 == FS_ATTN_PATH_WHOLE1 &&
                  (int)fs::AttnPath::kWhole2 == FS_ATTN_PATH_WHOLE2 && (int)fs::AttnPath::kWhole4 == FS_ATTN_PATH_WHOLE4,
              "the tuning values name the decompositions");

bool capturing(hipStream_t s) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &st) == hipSuccess && st != hipStreamCaptureStatusNone;
}

// A call whose kernels exchange tagged records through the workspace tells
// its own records from older ones by a tag.  Eager calls get a host epoch.
// Under stream capture an epoch would be frozen into the graph, and a
// replay could take the previous replay's records for its own, so a
// captured call passes 0: its kernels then tag by per-row counters kept in
// the workspace, which advance on the device at every replay.
unsigned long long call_epoch(hipStream_t s) {
    return capturing(s) ? 0ull : next_epoch();
}

// Decomposition of an attention call of n_bh rows over S keys (plus a
// generated-token job); chosen once per call.
fs::AttnPath attn_path_for(int n_bh, int S, int D, int esize, bool gen_job) {
    const int C = fs::cross_attn_chunk_keys(D, esize);
    const int NC = std::max(1, (S + C - 1) / C);
    return fs::choose_attn_path(n_bh, NC + (gen_job ? 1 : 0));
}

// FS_VALIDATE's check of the device-resident lengths: a synchronous copy to
// the host, refused while the stream is capturing (the copy and the
// synchronisation would end the capture).
int validate_lengths(const int32_t *len, int B, int limit, hipStream_t s, const char *what) {
    if (capturing(s))
        return fail(FS_ERR_UNSUPPORTED, "FS_VALIDATE copies %s to the host, which a capturing stream cannot do", what);
    std::vector<int32_t> lens((size_t)B);
    hipError_t e = hipMemcpyAsync(lens.data(), len, (size_t)B * 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(FS_ERR_HIP, "FS_VALIDATE copy of %s: %s (%d)", what, hipGetErrorString(e), (int)e);
    for (int b = 0; b < B; ++b)
        if (lens[b] < 0 || lens[b] > limit)
            return fail(FS_ERR_INVALID_ARG, "%s[%d] = %d outside [0, %d]", what, b, lens[b], limit);
    return FS_OK;
}

// Host-side shape checks shared by the workspace query and the launch.
// Returns FS_OK or an error status with g_last_error set.
int check_attn_sizes(int B, int k, int H, int S, int D, int dtype) {
    if (B < 0 || k < 0 || H < 0 || S < 0 || D < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (B=%d k=%d H=%d S=%d D=%d)", B, k, H, S, D);
    if (dtype != FS_F32 && dtype != FS_BF16)
        return fail(FS_ERR_UNSUPPORTED, "dtype %d is not FS_F32 or FS_BF16", dtype);
    if (!supported_d(D)) return fail(FS_ERR_UNSUPPORTED, "head dim D=%d not in {16,32,64,128}", D);
    if (k > 8) return fail(FS_ERR_UNSUPPORTED, "beam size k=%d > 8", k);
    const int esize = dtype == FS_BF16 ? 2 : 4;
    const long long C = fs::cross_attn_chunk_keys(D, esize);
    const long long nc = std::max(1LL, (S + C - 1) / C);
    const long long bh_padded = ((long long)B * H + 7) / 8 * 8;  // chunk grid is padded to 8 XCDs
    if ((long long)B * k * H > INT_MAX || bh_padded * (nc + 2) + (long long)B * k > INT_MAX)
        return fail(FS_ERR_INVALID_ARG, "problem too large for one launch (B=%d k=%d H=%d S=%d)",
                    B, k, H, S);
    // one (source, head) block of K or V is read through a 32-bit byte range
    if ((long long)S * D * esize > kMaxBlockBytes)
        return fail(FS_ERR_UNSUPPORTED, "one (source, head) block of S*D = %lld elements exceeds 2 GiB",
                    (long long)S * D);
    return FS_OK;
}

// Checks of fs_beam_cross_attn's arguments (also the attention half of the
// fused decode step); FS_OK or an error with g_last_error set.
int check_cross_attn(const void *q, const void *K, const void *V, const int32_t *src_len, void *out, int B,
                     int k, int H, int S, int D, int dtype, void *workspace, size_t workspace_bytes,
                     bool own_scratch = false) {
    const size_t esize = dtype == FS_BF16 ? 2 : 4;
    const size_t q_bytes = (size_t)B * k * H * D * esize;
    const size_t kv_bytes = (size_t)B * H * S * D * esize;
    if (!q || !out || !src_len || (kv_bytes > 0 && (!K || !V)))
        return fail(FS_ERR_INVALID_ARG, "null pointer (q=%p K=%p V=%p src_len=%p out=%p)",
                    q, K, V, (const void *)src_len, out);
    if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16))
        return fail(FS_ERR_INVALID_ARG, "q, K, V and out must be 16-byte aligned");
    if (!aligned(src_len, 4)) return fail(FS_ERR_INVALID_ARG, "src_len must be 4-byte aligned");
    if (overlaps(out, q_bytes, q, q_bytes) || overlaps(out, q_bytes, K, kv_bytes) ||
        overlaps(out, q_bytes, V, kv_bytes) || overlaps(out, q_bytes, src_len, (size_t)B * 4))
        return fail(FS_ERR_INVALID_ARG, "out overlaps an input");
    if (own_scratch) return FS_OK;   // the library's own array: sized and checked by the caller
    const size_t need = fs::cross_attn_workspace_floats(B, k, H, S, D, (int)esize, false) * sizeof(float);
    if (workspace_bytes < need || (need > 0 && !workspace))
        return fail(FS_ERR_INVALID_ARG, "workspace of %zu bytes at %p; %zu bytes needed",
                    workspace_bytes, workspace, need);
    if (!aligned(workspace, 16)) return fail(FS_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (need > 0 && (overlaps(workspace, need, q, q_bytes) || overlaps(workspace, need, K, kv_bytes) ||
                     overlaps(workspace, need, V, kv_bytes) || overlaps(workspace, need, out, q_bytes) ||
                     overlaps(workspace, need, src_len, (size_t)B * 4)))
        return fail(FS_ERR_INVALID_ARG, "workspace overlaps an argument");
    return FS_OK;
}

// Checks of fs_ngram_block's arguments that do not depend on the work being
// empty; FS_OK or an error with g_last_error set.
int check_ngram_sizes(int ld_tokens, int rows, int t, int n, int V) {
    if (rows < 0 || t < 0 || V < 0 || ld_tokens < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (rows=%d t=%d V=%d ld=%d)", rows, t, V, ld_tokens);
    if (n < 1) return fail(FS_ERR_INVALID_ARG, "n=%d < 1", n);
    if (ld_tokens < t) return fail(FS_ERR_INVALID_ARG, "ld_tokens=%d < t=%d", ld_tokens, t);
    return FS_OK;
}

// Checks of the n-gram buffers when there is work (rows > 0, t >= n).
int check_ngram_buffers(const int32_t *tokens, int ld_tokens, int rows, int t, const float *logits, int V) {
    if (!tokens || (V > 0 && !logits))
        return fail(FS_ERR_INVALID_ARG, "null pointer (tokens=%p logits=%p)", (const void *)tokens,
                    (const void *)logits);
    if (!aligned(tokens, 4) || !aligned(logits, 4))
        return fail(FS_ERR_INVALID_ARG, "tokens and logits must be 4-byte aligned");
    const size_t tok_bytes = ((size_t)(rows - 1) * ld_tokens + t) * 4;
    const size_t lg_bytes = (size_t)rows * V * 4;
    if (overlaps(tokens, tok_bytes, logits, lg_bytes))
        return fail(FS_ERR_INVALID_ARG, "logits overlap tokens");
    return FS_OK;
}

}  // namespace

extern "C" {

int fs_abi_version(void) { return FS_ABI_VERSION; }

const char *fs_status_string(int status) {
    switch (status) {
    case FS_OK: return "FS_OK";
    case FS_ERR_INVALID_ARG: return "FS_ERR_INVALID_ARG";
    case FS_ERR_UNSUPPORTED: return "FS_ERR_UNSUPPORTED";
    case FS_ERR_HIP: return "FS_ERR_HIP";
    default: return "unknown status";
    }
}

const char *fs_last_error(void) { return g_last_error.c_str(); }

size_t fs_beam_cross_attn_workspace_bytes(int B, int k, int H, int S, int D, int dtype) {
    g_last_error.clear();
    if (check_attn_sizes(B, k, H, S, D, dtype) != FS_OK) return (size_t)-1;
    if (B == 0 || k == 0 || H == 0) return 0;
    const int esize = dtype == FS_BF16 ? 2 : 4;
    return fs::cross_attn_workspace_floats(B, k, H, S, D, esize, false) * sizeof(float);
}

size_t fs_beam_prefix_attn_workspace_bytes(int B, int k, int H, int N, int T, int D, int dtype) {
    g_last_error.clear();
    if (T < 0) {
        fail(FS_ERR_INVALID_ARG, "negative size (T=%d)", T);
        return (size_t)-1;
    }
    if (check_attn_sizes(B, k, H, N, D, dtype) != FS_OK) return (size_t)-1;
    if (B == 0 || k == 0 || H == 0) return 0;
    const int esize = dtype == FS_BF16 ? 2 : 4;
    return fs::cross_attn_workspace_floats(B, k, H, N, D, esize, true) * sizeof(float);
}

int fs_beam_cross_attn(const void *q, const void *K, const void *V, const int32_t *src_len,
                       void *out, int B, int k, int H, int S, int D, int dtype,
                       void *workspace, size_t workspace_bytes, void *stream)
{
    g_last_error.clear();
    int st = check_attn_sizes(B, k, H, S, D, dtype);
    if (st != FS_OK) return st;
    if (B == 0 || k == 0 || H == 0) return FS_OK;
    st = check_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype, workspace, workspace_bytes);
    if (st != FS_OK) return st;

    hipStream_t s = static_cast<hipStream_t>(stream);
    const int esize = dtype == FS_BF16 ? 2 : 4;
    const fs::AttnPath path = attn_path_for(B * H, S, D, esize, false);
    if (validate_mode() && (st = validate_lengths(src_len, B, S, s, "src_len")) != FS_OK) return st;
    hipError_t e = fs::launch_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype == FS_BF16,
                                         static_cast<float *>(workspace), call_epoch(s), s, path);
    if (e != hipSuccess) return hip_fail(e, "fs_beam_cross_attn launch");
    return FS_OK;
}

}  // extern "C"

namespace {

// ---- the decode step without a caller workspace ---------------------------
// The split-KV decomposition keeps its partial records in `scratch`, one
// file-scope array per GPU, instead of a workspace the caller allocates.  In
// host code `scratch` only names the symbol: its device address, different
// on every GPU, comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = FS_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

__global__ void scratch_clear_kernel(uint4 *p, size_t n16) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

struct ScratchSlot {
    void *ptr = nullptr;   // device address of `scratch` on this device
    bool cleared = false;  // a clear has been enqueued before the first use
};
std::mutex g_scratch_mu;
ScratchSlot g_scratch[kMaxDevices];

// The device address of `scratch` on the device of `s` (the current device
// for the null stream), found once per device with that device current; the
// first use on a device enqueues a clear on `s`, so the array starts at zero.
int scratch_on(hipStream_t s, void **ptr) {
    int dev = -1;
    hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "fs_beam_decode_step_noalloc: device of the stream");
    if (dev < 0 || dev >= kMaxDevices) return fail(FS_ERR_UNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchSlot &slot = g_scratch[dev];
    if (!slot.ptr) {
        int cur = -1;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return hip_fail(e, "hipGetDevice");
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "hipSetDevice");
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess || !p) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        slot.ptr = p;
    }
    if (!slot.cleared) {
        hipLaunchKernelGGL(scratch_clear_kernel, dim3(256), dim3(256), 0, s, static_cast<uint4 *>(slot.ptr),
                           kScratchBytes / 16);
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "clear of the scratch array");
        slot.cleared = true;
    }
    *ptr = slot.ptr;
    return FS_OK;
}

// fs_beam_decode_step, with the caller's workspace (noalloc == false) or the
// scratch array (noalloc == true, workspace arguments ignored).
int decode_step(const void *q, const void *K, const void *V, const int32_t *src_len, void *out, int B, int k,
                int H, int S, int D, int dtype, const int32_t *tokens, int ld_tokens, int t, int n, float *logits,
                int vocab, void *workspace, size_t workspace_bytes, void *stream, bool noalloc)
{
    g_last_error.clear();
    int st = check_attn_sizes(B, k, H, S, D, dtype);
    if (st != FS_OK) return st;
    const long long rows_ll = (long long)B * k;
    if ((st = check_ngram_sizes(ld_tokens, (int)std::min<long long>(rows_ll, INT_MAX), t, n, vocab)) != FS_OK)
        return st;
    const int rows = (int)rows_ll;
    const bool attn = B > 0 && k > 0 && H > 0;
    const bool ngram = rows > 0 && t >= n && vocab > 0;
    const int esize_i = dtype == FS_BF16 ? 2 : 4;
    const fs::AttnPath path = attn ? attn_path_for(B * H, S, D, esize_i, false) : fs::AttnPath::kAuto;
    if (noalloc) {
        // only the split-KV form keeps records; its need must fit the array
        const size_t need = path == fs::AttnPath::kSplit
            ? fs::cross_attn_workspace_floats(B, k, H, S, D, esize_i, false) * sizeof(float) : 0;
        if (need > kScratchBytes)
            return fail(FS_ERR_UNSUPPORTED, "fs_beam_decode_step_noalloc: %d rows take the split-KV form, whose "
                        "%zu bytes of partial records exceed the %zu-byte scratch array", B * H, need, kScratchBytes);
        workspace = nullptr;
        workspace_bytes = need;
    }
    if (attn && (st = check_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype, noalloc ? nullptr : workspace,
                                       noalloc ? 0 : workspace_bytes, noalloc)) != FS_OK)
        return st;
    if (ngram) {
        if ((st = check_ngram_buffers(tokens, ld_tokens, rows, t, logits, vocab)) != FS_OK) return st;
        if (attn) {
            // the two halves write disjoint buffers and read none of the other's outputs
            const size_t esize = dtype == FS_BF16 ? 2 : 4;
            const size_t q_bytes = (size_t)B * k * H * D * esize, kv_bytes = (size_t)B * H * S * D * esize;
            const size_t lg_bytes = (size_t)rows * vocab * 4;
            const size_t tok_bytes = ((size_t)(rows - 1) * ld_tokens + t) * 4;
            const size_t ws_bytes = noalloc ? 0
                : fs::cross_attn_workspace_floats(B, k, H, S, D, (int)esize, false) * sizeof(float);
            if (overlaps(logits, lg_bytes, q, q_bytes) || overlaps(logits, lg_bytes, K, kv_bytes) ||
                overlaps(logits, lg_bytes, V, kv_bytes) || overlaps(logits, lg_bytes, out, q_bytes) ||
                overlaps(logits, lg_bytes, src_len, (size_t)B * 4) || overlaps(logits, lg_bytes, workspace, ws_bytes))
                return fail(FS_ERR_INVALID_ARG, "logits overlap an attention argument");
            if (overlaps(tokens, tok_bytes, out, q_bytes) || overlaps(tokens, tok_bytes, workspace, ws_bytes))
                return fail(FS_ERR_INVALID_ARG, "tokens overlap out or the workspace");
        }
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!attn) {
        if (!ngram) return FS_OK;
        hipError_t e = fs::launch_ngram_block(tokens, ld_tokens, rows, t, n, logits, vocab, s);
        if (e != hipSuccess) return hip_fail(e, "fs_beam_decode_step n-gram launch");
        return FS_OK;
    }
    if (validate_mode() && (st = validate_lengths(src_len, B, S, s, "src_len")) != FS_OK) return st;
    if (noalloc && path == fs::AttnPath::kSplit && (st = scratch_on(s, &workspace)) != FS_OK) return st;
    const fs::NgramRows ng{tokens, ld_tokens, rows, t, n, logits, vocab};
    hipError_t e = fs::launch_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype == FS_BF16,
                                         static_cast<float *>(workspace), call_epoch(s), s, path,
                                         ngram ? &ng : nullptr);
    if (e != hipSuccess) return hip_fail(e, noalloc ? "fs_beam_decode_step_noalloc launch" : "fs_beam_decode_step launch");
    return FS_OK;
}

}  // namespace

extern "C" {

int fs_beam_decode_step(const void *q, const void *K, const void *V, const int32_t *src_len, void *out,
                        int B, int k, int H, int S, int D, int dtype,
                        const int32_t *tokens, int ld_tokens, int t, int n, float *logits, int vocab,
                        void *workspace, size_t workspace_bytes, void *stream)
{
    return decode_step(q, K, V, src_len, out, B, k, H, S, D, dtype, tokens, ld_tokens, t, n, logits, vocab,
                       workspace, workspace_bytes, stream, false);
}

int fs_beam_decode_step_noalloc(const void *q, const void *K, const void *V, const int32_t *src_len, void *out,
                                int B, int k, int H, int S, int D, int dtype,
                                const int32_t *tokens, int ld_tokens, int t, int n, float *logits, int vocab,
                                void *stream)
{
    return decode_step(q, K, V, src_len, out, B, k, H, S, D, dtype, tokens, ld_tokens, t, n, logits, vocab,
                       nullptr, 0, stream, true);
}

int fs_trace_set(void *buffer, size_t bytes)
{
    g_last_error.clear();
    if (bytes > 0 && !buffer) return fail(FS_ERR_INVALID_ARG, "null trace buffer of %zu bytes", bytes);
    if (buffer && !aligned(buffer, 8)) return fail(FS_ERR_INVALID_ARG, "trace buffer must be 8-byte aligned");
    const size_t cap = buffer ? bytes / 64 : 0;
    unsigned long long *buf = cap ? static_cast<unsigned long long *>(buffer) : nullptr;
    const unsigned int c = cap > 0xffffffffu ? 0xffffffffu : (unsigned int)cap;
    hipError_t e = fs::set_attn_trace(buf, c);
    if (e == hipErrorNotSupported)
        return fail(FS_ERR_UNSUPPORTED, "this library was built without workgroup tracing (build with trace=True)");
    if (e == hipSuccess) e = fs::set_select_trace(buf, c);
    if (e != hipSuccess) return hip_fail(e, "fs_trace_set");
    return FS_OK;
}

int fs_set_tuning(int knob, int value)
{
    switch (knob) {
    case FS_TUNE_ATTN_PATH:
        if (value < 0 || value > FS_ATTN_PATH_WHOLE4) return -1;
        return static_cast<int>(fs::set_attn_path_override(static_cast<fs::AttnPath>(value)));
    case FS_TUNE_SELECT_SLICES:
        if (value < 0) return -1;
        return fs::set_select_slices_override(value);
    case FS_TUNE_VALIDATE: {
        if (value != 0 && value != 1) return -1;
        const int prev = validate_mode() ? 1 : 0;
        g_validate.store(value, std::memory_order_relaxed);
        return prev;
    }
    default:
        return -1;
    }
}

}  // extern "C"

namespace {

// Both split-cache entry points: without (anc == null) and with the
// ancestry table of the generated rows.
int prefix_attn(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len, const void *Kt,
                const void *Vt, const int32_t *anc, int ld_anc, int T, int t, void *out, int B, int k, int H, int N,
                int D, int dtype, void *workspace, size_t workspace_bytes, void *stream, bool indirect)
{
    g_last_error.clear();
    if (T < 0 || t < 0) return fail(FS_ERR_INVALID_ARG, "negative size (T=%d t=%d)", T, t);
    if (t > T) return fail(FS_ERR_INVALID_ARG, "t=%d exceeds the generated-token capacity T=%d", t, T);
    int st = check_attn_sizes(B, k, H, N, D, dtype);
    if (st != FS_OK) return st;
    if (B == 0 || k == 0 || H == 0) return FS_OK;

    const size_t esize = dtype == FS_BF16 ? 2 : 4;
    const size_t q_bytes = (size_t)B * k * H * D * esize;
    const size_t p_bytes = (size_t)B * H * N * D * esize;
    const size_t g_bytes = (size_t)B * k * H * T * D * esize;
    if (!q || !out || !prefix_len || (p_bytes > 0 && (!Kp || !Vp)) || (g_bytes > 0 && (!Kt || !Vt)))
        return fail(FS_ERR_INVALID_ARG, "null pointer (q=%p Kp=%p Vp=%p prefix_len=%p Kt=%p Vt=%p out=%p)",
                    q, Kp, Vp, (const void *)prefix_len, Kt, Vt, out);
    if (!aligned(q, 16) || !aligned(Kp, 16) || !aligned(Vp, 16) || !aligned(Kt, 16) || !aligned(Vt, 16) ||
        !aligned(out, 16))
        return fail(FS_ERR_INVALID_ARG, "q, Kp, Vp, Kt, Vt and out must be 16-byte aligned");
    if (!aligned(prefix_len, 4)) return fail(FS_ERR_INVALID_ARG, "prefix_len must be 4-byte aligned");
    if (overlaps(out, q_bytes, q, q_bytes) || overlaps(out, q_bytes, Kp, p_bytes) ||
        overlaps(out, q_bytes, Vp, p_bytes) || overlaps(out, q_bytes, Kt, g_bytes) ||
        overlaps(out, q_bytes, Vt, g_bytes) || overlaps(out, q_bytes, prefix_len, (size_t)B * 4))
        return fail(FS_ERR_INVALID_ARG, "out overlaps an input");
    if ((long long)B * k * H * ((long long)T * D) > (long long)INT_MAX * 16)
        return fail(FS_ERR_INVALID_ARG, "generated-token cache too large");
    if ((long long)T * D * (long long)esize > kMaxBlockBytes)
        return fail(FS_ERR_UNSUPPORTED, "one (hypothesis, head) block of T*D = %lld generated elements exceeds 2 GiB",
                    (long long)T * D);
    if (indirect && t > 0) {
        if (!anc) return fail(FS_ERR_INVALID_ARG, "null ancestry table with t=%d > 0", t);
        if (ld_anc < t) return fail(FS_ERR_INVALID_ARG, "ld_anc=%d < t=%d", ld_anc, t);
        if (!aligned(anc, 4)) return fail(FS_ERR_INVALID_ARG, "anc must be 4-byte aligned");
        // the rows of a source's k beams are read through one buffer range
        if ((long long)k * H * T * D * (long long)esize > 0x7ff00000LL)
            return fail(FS_ERR_UNSUPPORTED, "a source's generated-token cache exceeds 2 GiB (k=%d H=%d T=%d D=%d)",
                        k, H, T, D);
        if (overlaps(out, q_bytes, anc, ((size_t)(B * k - 1) * ld_anc + t) * 4))
            return fail(FS_ERR_INVALID_ARG, "out overlaps the ancestry table");
    }
    const size_t need = fs_beam_prefix_attn_workspace_bytes(B, k, H, N, T, D, dtype);
    if (workspace_bytes < need || (need > 0 && !workspace))
        return fail(FS_ERR_INVALID_ARG, "workspace of %zu bytes at %p; %zu bytes needed",
                    workspace_bytes, workspace, need);
    if (!aligned(workspace, 16)) return fail(FS_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (need > 0 && (overlaps(workspace, need, q, q_bytes) || overlaps(workspace, need, Kp, p_bytes) ||
                     overlaps(workspace, need, Vp, p_bytes) || overlaps(workspace, need, Kt, g_bytes) ||
                     overlaps(workspace, need, Vt, g_bytes) || overlaps(workspace, need, out, q_bytes) ||
                     overlaps(workspace, need, prefix_len, (size_t)B * 4)))
        return fail(FS_ERR_INVALID_ARG, "workspace overlaps an argument");

    hipStream_t s = static_cast<hipStream_t>(stream);
    const fs::AttnPath path = attn_path_for(B * H, N, D, dtype == FS_BF16 ? 2 : 4, t > 0);
    if (validate_mode() && (st = validate_lengths(prefix_len, B, N, s, "prefix_len")) != FS_OK) return st;
    hipError_t e = fs::launch_prefix_attn(q, Kp, Vp, prefix_len, Kt, Vt, T, t, indirect && t > 0 ? anc : nullptr,
                                          ld_anc, out, B, k, H, N, D, dtype == FS_BF16,
                                          static_cast<float *>(workspace), call_epoch(s), s, path);
    if (e != hipSuccess) return hip_fail(e, indirect ? "fs_beam_prefix_attn_indirect launch" : "fs_beam_prefix_attn launch");
    return FS_OK;
}

}  // namespace

extern "C" {

int fs_beam_prefix_attn(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                        const void *Kt, const void *Vt, int T, int t, void *out,
                        int B, int k, int H, int N, int D, int dtype,
                        void *workspace, size_t workspace_bytes, void *stream)
{
    return prefix_attn(q, Kp, Vp, prefix_len, Kt, Vt, nullptr, 0, T, t, out, B, k, H, N, D, dtype, workspace,
                       workspace_bytes, stream, false);
}

int fs_beam_prefix_attn_indirect(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                                 const void *Kt, const void *Vt, const int32_t *anc, int ld_anc, int T, int t,
                                 void *out, int B, int k, int H, int N, int D, int dtype, void *workspace,
                                 size_t workspace_bytes, void *stream)
{
    return prefix_attn(q, Kp, Vp, prefix_len, Kt, Vt, anc, ld_anc, T, t, out, B, k, H, N, D, dtype, workspace,
                       workspace_bytes, stream, true);
}

int fs_beam_ancestry_step(int32_t *anc, int ld_anc, const int32_t *parent, int B, int k, int t, void *stream)
{
    g_last_error.clear();
    if (B < 0 || k < 0 || t < 0 || ld_anc < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (B=%d k=%d t=%d ld_anc=%d)", B, k, t, ld_anc);
    if (k < 1 || k > 16) return fail(FS_ERR_UNSUPPORTED, "beam size k=%d outside [1, 16]", k);
    if (t >= ld_anc) return fail(FS_ERR_INVALID_ARG, "column t=%d does not exist (ld_anc=%d)", t, ld_anc);
    if (B == 0) return FS_OK;
    if (!anc || !parent) return fail(FS_ERR_INVALID_ARG, "null pointer (anc=%p parent=%p)", (void *)anc,
                                     (const void *)parent);
    if (!aligned(anc, 4) || !aligned(parent, 4)) return fail(FS_ERR_INVALID_ARG, "anc and parent must be 4-byte aligned");
    if ((long long)B * k * ld_anc > (long long)INT_MAX * 4)
        return fail(FS_ERR_UNSUPPORTED, "ancestry table too large (B=%d k=%d ld_anc=%d)", B, k, ld_anc);
    if (overlaps(anc, (size_t)B * k * ld_anc * 4, parent, (size_t)B * k * 4))
        return fail(FS_ERR_INVALID_ARG, "parent overlaps the ancestry table");
    hipError_t e = fs::launch_ancestry_step(anc, ld_anc, parent, B, k, t, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "fs_beam_ancestry_step launch");
    return FS_OK;
}

int fs_ngram_block(const int32_t *tokens, int ld_tokens, int rows, int t, int n,
                   float *logits, int V, void *stream)
{
    g_last_error.clear();
    int st = check_ngram_sizes(ld_tokens, rows, t, n, V);
    if (st != FS_OK) return st;
    if (rows == 0 || t < n) return FS_OK;  // no window: nothing to ban
    if ((st = check_ngram_buffers(tokens, ld_tokens, rows, t, logits, V)) != FS_OK) return st;
    if (V == 0) return FS_OK;  // no id is in range: nothing can be written
    hipError_t e = fs::launch_ngram_block(tokens, ld_tokens, rows, t, n, logits, V,
                                          static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "fs_ngram_block launch");
    return FS_OK;
}

}  // extern "C"

namespace {

int check_select_sizes(int B, int k, int V, int c) {
    if (B < 0 || k < 0 || V < 0 || c < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (B=%d k=%d V=%d c=%d)", B, k, V, c);
    if (k < 1 || k > 16) return fail(FS_ERR_UNSUPPORTED, "beam size k=%d outside [1, 16]", k);
    if (V < 1) return fail(FS_ERR_INVALID_ARG, "vocabulary V=%d < 1", V);
    if (c < 1 || c > 16) return fail(FS_ERR_UNSUPPORTED, "c=%d outside [1, 16]", c);
    if ((long long)c > (long long)k * V) return fail(FS_ERR_INVALID_ARG, "c=%d > k*V=%lld", c, (long long)k * V);
    if ((long long)k * V > 0xffffffffLL) return fail(FS_ERR_UNSUPPORTED, "k*V=%lld flat indices exceed 32 bits",
                                                     (long long)k * V);
    const long long rows = (long long)B * k;
    if (rows > INT_MAX) return fail(FS_ERR_INVALID_ARG, "B*k=%lld too large", rows);
    const int ns = fs::beam_select_slices((int)rows, V, k, c);
    if ((long long)k * ns * c > fs::beam_select_max_candidates())
        return fail(FS_ERR_UNSUPPORTED, "k*slices*c=%lld candidates per source exceed %d", (long long)k * ns * c,
                    fs::beam_select_max_candidates());
    if ((long long)k * ns * (2 + 2 * c) > fs::beam_select_max_record_words())
        return fail(FS_ERR_UNSUPPORTED, "k*slices*(2+2c)=%lld record words per source exceed %d",
                    (long long)k * ns * (2 + 2 * c), fs::beam_select_max_record_words());
    if (rows * ns + B > INT_MAX) return fail(FS_ERR_INVALID_ARG, "problem too large for one launch");
    return FS_OK;
}

}  // namespace

extern "C" {

size_t fs_beam_select_workspace_bytes(int B, int k, int V, int c) {
    g_last_error.clear();
    if (check_select_sizes(B, k, V, c) != FS_OK) return (size_t)-1;
    if (B == 0) return 0;
    return fs::beam_select_workspace_words(B, k, V, c) * 8;
}

int fs_beam_select(const float *logits, const float *beam_scores, const int32_t *tokens, int ld_tokens,
                   int t, int n, float *out_scores, int32_t *out_beam, int32_t *out_token,
                   int B, int k, int V, int c, void *workspace, size_t workspace_bytes, void *stream)
{
    g_last_error.clear();
    int st = check_select_sizes(B, k, V, c);
    if (st != FS_OK) return st;
    if (n < 0 || t < 0 || ld_tokens < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (n=%d t=%d ld_tokens=%d)", n, t, ld_tokens);
    if (n > 0 && ld_tokens < t) return fail(FS_ERR_INVALID_ARG, "ld_tokens=%d < t=%d", ld_tokens, t);
    if (B == 0) return FS_OK;
    const bool need_tokens = n > 0 && t >= n;
    if (!logits || !beam_scores || !out_scores || !out_beam || !out_token || (need_tokens && !tokens))
        return fail(FS_ERR_INVALID_ARG, "null pointer (logits=%p beam_scores=%p tokens=%p outputs=%p %p %p)",
                    (const void *)logits, (const void *)beam_scores, (const void *)tokens, (void *)out_scores,
                    (void *)out_beam, (void *)out_token);
    if (!aligned(logits, 4) || !aligned(beam_scores, 4) || !aligned(tokens, 4) || !aligned(out_scores, 4) ||
        !aligned(out_beam, 4) || !aligned(out_token, 4))
        return fail(FS_ERR_INVALID_ARG, "arrays must be 4-byte aligned");
    const size_t rows = (size_t)B * k;
    const size_t lg_bytes = rows * V * 4, bs_bytes = rows * 4, o_bytes = (size_t)B * c * 4;
    const size_t tok_bytes = need_tokens ? ((rows - 1) * ld_tokens + t) * 4 : 0;
    const void *outs[3] = {out_scores, out_beam, out_token};
    for (int i = 0; i < 3; ++i) {
        if (overlaps(outs[i], o_bytes, logits, lg_bytes) || overlaps(outs[i], o_bytes, beam_scores, bs_bytes) ||
            overlaps(outs[i], o_bytes, tokens, tok_bytes))
            return fail(FS_ERR_INVALID_ARG, "an output overlaps an input");
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i], o_bytes, outs[j], o_bytes)) return fail(FS_ERR_INVALID_ARG, "outputs overlap");
    }
    const size_t need = fs_beam_select_workspace_bytes(B, k, V, c);
    if (workspace_bytes < need || !workspace)
        return fail(FS_ERR_INVALID_ARG, "workspace of %zu bytes at %p; %zu bytes needed", workspace_bytes,
                    workspace, need);
    if (!aligned(workspace, 16)) return fail(FS_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (overlaps(workspace, need, logits, lg_bytes) || overlaps(workspace, need, beam_scores, bs_bytes) ||
        overlaps(workspace, need, tokens, tok_bytes) || overlaps(workspace, need, out_scores, o_bytes) ||
        overlaps(workspace, need, out_beam, o_bytes) || overlaps(workspace, need, out_token, o_bytes))
        return fail(FS_ERR_INVALID_ARG, "workspace overlaps an argument");
    hipError_t e = fs::launch_beam_select(logits, beam_scores, need_tokens ? tokens : nullptr, ld_tokens, t,
                                          need_tokens ? n : 0, out_scores, out_beam, out_token, B, k, V, c,
                                          static_cast<unsigned long long *>(workspace),
                                          call_epoch(static_cast<hipStream_t>(stream)),
                                          static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "fs_beam_select launch");
    return FS_OK;
}


int fs_cache_reorder(void *K, void *V, const int32_t *parent, int B, int k, int H, int T, int t, int D, int dtype,
                     void *stream)
{
    g_last_error.clear();
    if (B < 0 || k < 0 || H < 0 || T < 0 || t < 0 || D < 0)
        return fail(FS_ERR_INVALID_ARG, "negative size (B=%d k=%d H=%d T=%d t=%d D=%d)", B, k, H, T, t, D);
    if (t > T) return fail(FS_ERR_INVALID_ARG, "t=%d > T=%d", t, T);
    if (dtype != FS_F32 && dtype != FS_BF16)
        return fail(FS_ERR_UNSUPPORTED, "dtype %d is not FS_F32 or FS_BF16", dtype);
    if (k < 1 || k > 16) return fail(FS_ERR_UNSUPPORTED, "beam size k=%d outside [1, 16]", k);
    const int esize = dtype == FS_BF16 ? 2 : 4;
    if (((long long)D * esize) % 4 != 0)
        return fail(FS_ERR_UNSUPPORTED, "a row of D=%d elements is not a whole number of 4-byte words", D);
    if (B == 0 || H == 0 || t == 0 || D == 0) return FS_OK;  // nothing moves
    if (!K || !parent) return fail(FS_ERR_INVALID_ARG, "null pointer (K=%p parent=%p)", K, (const void *)parent);
    if (!aligned(K, 4) || !aligned(V, 4) || !aligned(parent, 4))
        return fail(FS_ERR_INVALID_ARG, "K, V and parent must be 4-byte aligned");
    const long long beam_bytes = (long long)H * T * D * esize;
    if ((long long)k * beam_bytes > INT_MAX || (long long)t * D * esize > INT_MAX ||
        (long long)2 * B * H * (((long long)t * D * esize / 4 + 255) / 256) > UINT_MAX)
        return fail(FS_ERR_UNSUPPORTED, "cache too large for one launch (B=%d k=%d H=%d T=%d D=%d)", B, k, H, T, D);
    const size_t cache_bytes = (size_t)B * k * beam_bytes;
    if (overlaps(K, cache_bytes, V, V ? cache_bytes : 0)) return fail(FS_ERR_INVALID_ARG, "K overlaps V");
    if (overlaps(K, cache_bytes, parent, (size_t)B * k * 4) || overlaps(V, V ? cache_bytes : 0, parent, (size_t)B * k * 4))
        return fail(FS_ERR_INVALID_ARG, "parent overlaps the cache");
    hipError_t e = fs::launch_cache_reorder(K, V, parent, B, k, H, T, t, D, esize, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "fs_cache_reorder launch");
    return FS_OK;
}

}  // extern "C"
