// Per-beam cache reorder for gfx950, in place.
//
// After a beam-search selection step the new hypothesis j of source b
// continues the old hypothesis parent[b*k + j] of the same source (Section
// 2.2, cache maintenance).  Its cache of generated tokens must then hold what
// that parent's held: for every head h and position tau < t,
//     cache[b*k + j, h, tau, :] = old cache[b*k + parent[b*k + j], h, tau, :].
// With the cache split (Section 4.1.1) only this per-beam part is reordered;
// the prefix and encoder caches are shared by the beams and never move.
//
// Bound by HBM bandwidth.  One lane owns one chunk (16 or 4 bytes) of the
// [t, D] block of one (source, head) for all k beams: it loads that chunk of
// every beam some other beam continues, waits for all its loads, then
// stores the chunk of every beam whose parent is another beam.  No other
// lane touches these bytes, so the copy is in place without a barrier or a
// second buffer, and beams that continue themselves are neither read nor
// written.
#include <stdint.h>

#include "launch.h"

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

namespace fs {
namespace {

constexpr int kThreads = 256;
// Loads and stores are non-temporal: each byte is touched once per call, and
// marking it so lets the caches stream it (about 15 % faster on MI355X).
constexpr int kNonTemporal = 2;

// Raw buffer resource over `bytes` bytes at p: accesses at or past the end
// read 0 and write nothing, without a memory access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *p, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, 0x00020000);
}

template <int CHUNK>
struct Chunk;
template <>
struct Chunk<16> {
    using T = u32x4_t;
    static __device__ T load(__amdgpu_buffer_rsrc_t r, int off) {
        return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
    }
    static __device__ void store(T v, __amdgpu_buffer_rsrc_t r, int off) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kNonTemporal);
    }
};
template <>
struct Chunk<4> {
    using T = uint32_t;
    static __device__ T load(__amdgpu_buffer_rsrc_t r, int off) {
        return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kNonTemporal);
    }
    static __device__ void store(T v, __amdgpu_buffer_rsrc_t r, int off) {
        __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, kNonTemporal);
    }
};

// One launch covers both tensors: block g is (tensor, source, head, block of
// chunks), chunks fastest.  `region` = t*D*esize, the used bytes of one
// (hypothesis, head) block.
template <int KMAX, int CHUNK>
__global__ __launch_bounds__(kThreads) void cache_reorder_kernel(unsigned char *K, unsigned char *V,
                                                                 const int32_t *parent, int B, int k, int H,
                                                                 long long beam_bytes, long long head_bytes,
                                                                 int region, int nblk)
{
    using C = Chunk<CHUNK>;
    int g = blockIdx.x;
    const int qb = g % nblk;
    g /= nblk;
    const int h = g % H;
    g /= H;
    const int b = g % B;
    unsigned char *cache = g / B ? V : K;
    const int off = (qb * kThreads + (int)threadIdx.x) * CHUNK;

    // parents of the source's beams (wave-uniform): kids[i] = the beams other
    // than i that continue beam i, needed = the beams with kids
    uint32_t kids[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) kids[i] = 0u;
    uint32_t needed = 0u;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
        if (j < k) {
            const int p = __builtin_amdgcn_readfirstlane(parent[(size_t)b * k + j]);
#pragma unroll
            for (int i = 0; i < KMAX; ++i) kids[i] |= (p == i && i != j) ? 1u << j : 0u;
            needed |= (p >= 0 && p < k && p != j) ? 1u << p : 0u;
        }
    }
    if (needed == 0u) return;
    unsigned char *blk = cache + (size_t)b * k * beam_bytes + (size_t)h * head_bytes;

    // a beam nobody continues gets an empty range: its load reads nothing
    typename C::T r[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
        r[i] = C::load(buf_rsrc(blk + (size_t)i * beam_bytes, ((needed >> i) & 1u) ? region : 0), off);
    // every load has returned before the first store: a store to a beam's
    // chunk never overtakes the read of that chunk
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
        if ((needed >> i) & 1u) {
#pragma unroll
            for (int j = 0; j < KMAX; ++j)
                if ((kids[i] >> j) & 1u) C::store(r[i], buf_rsrc(blk + (size_t)j * beam_bytes, region), off);
        }
    }
}

template <int CHUNK>
hipError_t launch_chunks(unsigned char *K, unsigned char *V, const int32_t *parent, int B, int k, int H,
                         long long beam_bytes, long long head_bytes, int region, hipStream_t stream)
{
    const int nq = region / CHUNK;
    const int nblk = (nq + kThreads - 1) / kThreads;
    const long long grid = (long long)(V ? 2 : 1) * B * H * nblk;
    const dim3 gd((unsigned)grid), bd(kThreads);
    if (k <= 4)
        hipLaunchKernelGGL((cache_reorder_kernel<4, CHUNK>), gd, bd, 0, stream, K, V, parent, B, k, H, beam_bytes,
                           head_bytes, region, nblk);
    else if (k <= 8)
        hipLaunchKernelGGL((cache_reorder_kernel<8, CHUNK>), gd, bd, 0, stream, K, V, parent, B, k, H, beam_bytes,
                           head_bytes, region, nblk);
    else
        hipLaunchKernelGGL((cache_reorder_kernel<16, CHUNK>), gd, bd, 0, stream, K, V, parent, B, k, H, beam_bytes,
                           head_bytes, region, nblk);
    return hipGetLastError();
}

// Ancestry step: block (source b, block of columns); lane tau owns column tau
// of the source's k rows.  Columns tau < t take the parent's entry, column t
// the beam's own index.  All loads come before all stores, so it is in place.
template <int KMAX>
__global__ __launch_bounds__(kThreads) void ancestry_step_kernel(int32_t *anc, int ld, const int32_t *parent, int k,
                                                                 int t, int nblk)
{
    const int b = blockIdx.x / nblk;
    const int tau = (blockIdx.x % nblk) * kThreads + (int)threadIdx.x;
    if (tau > t) return;
    int32_t *col = anc + (size_t)b * k * ld + tau;
    // the column's entries first: they do not depend on the parents, so both
    // sets of loads are in flight together
    int32_t v[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) v[i] = (i < k && tau < t) ? col[(size_t)i * ld] : 0;
    // the parents (wave-uniform), all loads issued before any is used
    int par[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) par[j] = j < k ? parent[(size_t)b * k + j] : j;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) par[j] = (par[j] >= 0 && par[j] < k) ? par[j] : j;
    if (tau < t) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): every load before the first store
#pragma unroll
        for (int j = 0; j < KMAX; ++j) {
            if (j < k && par[j] != j) {
                int32_t x = v[0];
#pragma unroll
                for (int i = 1; i < KMAX; ++i) x = par[j] == i ? v[i] : x;
                col[(size_t)j * ld] = x;
            }
        }
    } else {
#pragma unroll
        for (int j = 0; j < KMAX; ++j)
            if (j < k) col[(size_t)j * ld] = j;
    }
}

}  // namespace

hipError_t launch_ancestry_step(int32_t *anc, int ld, const int32_t *parent, int B, int k, int t,
                                hipStream_t stream)
{
    const int nblk = (t + 1 + kThreads - 1) / kThreads;
    const dim3 gd((unsigned)((long long)B * nblk)), bd(kThreads);
    if (k <= 4)
        hipLaunchKernelGGL(ancestry_step_kernel<4>, gd, bd, 0, stream, anc, ld, parent, k, t, nblk);
    else if (k <= 8)
        hipLaunchKernelGGL(ancestry_step_kernel<8>, gd, bd, 0, stream, anc, ld, parent, k, t, nblk);
    else
        hipLaunchKernelGGL(ancestry_step_kernel<16>, gd, bd, 0, stream, anc, ld, parent, k, t, nblk);
    return hipGetLastError();
}

int cache_reorder_chunk(const void *K, const void *V, int T, int t, int D, int esize) {
    // 16-byte chunks when every (hypothesis, head) block starts on a 16-byte
    // boundary and its t rows are a whole number of chunks
    const long long row = (long long)D * esize;
    const bool a16 = (reinterpret_cast<uintptr_t>(K) & 15) == 0 && (reinterpret_cast<uintptr_t>(V) & 15) == 0;
    return a16 && ((long long)T * row) % 16 == 0 && ((long long)t * row) % 16 == 0 ? 16 : 4;
}

hipError_t launch_cache_reorder(void *K, void *V, const int32_t *parent, int B, int k, int H, int T, int t, int D,
                                int esize, hipStream_t stream)
{
    const long long head_bytes = (long long)T * D * esize;
    const long long beam_bytes = head_bytes * H;
    const int chunk = cache_reorder_chunk(K, V, T, t, D, esize);
    const int region = (int)((long long)t * D * esize);
    auto *k8 = static_cast<unsigned char *>(K), *v8 = static_cast<unsigned char *>(V);
    return chunk == 16 ? launch_chunks<16>(k8, v8, parent, B, k, H, beam_bytes, head_bytes, region, stream)
                       : launch_chunks<4>(k8, v8, parent, B, k, H, beam_bytes, head_bytes, region, stream);
}

}  // namespace fs
