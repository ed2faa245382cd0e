// One beam-search selection step over the logits of a decode step, for gfx950.
//
// Beam search keeps, at every step, the best candidates of each source
// (Section 2.1 of the paper); the n-gram bans of Algorithm 1 (Section 4.2)
// give banned tokens zero probability.  For source b with hypotheses
// r = b*k + i and running log-probabilities beam_scores[r]:
//   lse_r = log sum_v exp(logits[r, v])            (every token)
//   cand(i*V + v) = beam_scores[r] + logits[r, v] - lse_r, or -inf if v is
//                   banned for row r
// and the c best candidates of the source are returned, best first, equal
// values in increasing flat index i*V + v.  The logits are read once and
// never written.
//
// One launch, bound by HBM bandwidth:
//   * one workgroup per (row, slice of the vocabulary): it issues all its
//     row loads first (16 bytes per lane and load), scans the row's history
//     for banned tokens into an LDS bitmap while they are in flight, then
//     takes each wave's (max, sum of exp) in two passes over registers, then
//     sets its banned values to -inf.  Its c best candidates come from a
//     threshold: the c-th largest of 64 block maxima (blocks of adjacent
//     lanes) has c distinct positions at or above it, so the c best of the
//     slice all lie there.  The few positions at or above it (about c for
//     random logits) are collected in LDS by ballots and ranked.  A slice
//     with too many positions at the threshold (equal logits) takes an exact
//     c-round selection instead.  The results go to the workspace as tagged
//     partial records;
//   * one merger workgroup per source, after all slice workgroups in the
//     grid, combines the slices' (max, sum) into each row's lse, scores the
//     k * slices * c candidates and keeps the c best.
// Each logit costs about five vector instructions (a max, a fused scale,
// an exp, an add and a compare), which keeps the slice pass under the time
// its bytes take to arrive.
// Candidates are compared as 64-bit keys (order-preserving bits of the value,
// then the complement of the flat index), so equal values resolve to the
// smaller index without a second comparison.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <atomic>


#include "launch.h"
#include "trace.h"

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

namespace fs {
namespace {

constexpr int kWave = 64;
constexpr int kThreads = 512;
constexpr int kPer = 32;                 // logits per thread and slice
constexpr int kSliceMax = kThreads * kPer;
constexpr int kCap = 1024;               // collected candidates per slice before the exact path
constexpr int kMergeCap = 1024;          // candidates a merger ranks: k * slices * c
constexpr int kMergeWords = 2048;        // record words a merger reads: k * slices * (2 + 2c)
constexpr int kMaxSpins = 1 << 14;       // bounded re-reads of a record word (about 10 ms)
constexpr int kNMax = 8;                 // n-gram sizes whose first window is loaded ahead
constexpr int kWaves = kThreads / kWave;
constexpr int kBlocks = kWave / kWaves;   // threshold blocks per wave: 64 in a workgroup

#if FS_TRACE
__device__ trace::Target g_trace{nullptr, 0};
#endif
// this workgroup's timeline words in a trace build, else null
__device__ __forceinline__ unsigned long long *trace_slot() {
#if FS_TRACE
    return trace::slot(g_trace);
#else
    return nullptr;
#endif
}

// Order-preserving 32-bit image of a float (larger value, larger image);
// -0 is taken as +0.
__device__ __forceinline__ uint32_t ordered(float x) {
    const uint32_t u = __float_as_uint(x + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unordered(uint32_t o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
// Candidate key: value first, then the smaller index.  0 is below every key.
__device__ __forceinline__ unsigned long long make_key(float x, uint32_t idx) {
    return ((unsigned long long)ordered(x) << 32) | (uint32_t)~idx;
}

// Cross-lane steps of a wave-wide reduction, all on the VALU: DPP inside
// rows of 16 lanes (quad permutes, then the half-row and row mirrors), then
// permlane swaps across the 16- and 32-lane halves.  After the six steps
// every lane has combined all 64 values, in the same order in every lane.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
template <int STEP>
__device__ __forceinline__ void partner(uint32_t &a, uint32_t &b, uint32_t x, uint32_t y) {
    // (a, b) = the (x, y) of this step's partner lane
    if constexpr (STEP == 0) { a = dpp_u32<0xB1>(x); b = dpp_u32<0xB1>(y); }        // quad_perm [1,0,3,2]
    else if constexpr (STEP == 1) { a = dpp_u32<0x4E>(x); b = dpp_u32<0x4E>(y); }   // quad_perm [2,3,0,1]
    else if constexpr (STEP == 2) { a = dpp_u32<0x141>(x); b = dpp_u32<0x141>(y); } // row_half_mirror
    else if constexpr (STEP == 3) { a = dpp_u32<0x140>(x); b = dpp_u32<0x140>(y); } // row_mirror
    else if constexpr (STEP == 4) {
        const auto rx = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        const auto ry = __builtin_amdgcn_permlane16_swap(y, y, false, false);
        const bool hi = __lane_id() & 16;
        a = hi ? rx[0] : rx[1];
        b = hi ? ry[0] : ry[1];
    } else {
        const auto rx = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        const auto ry = __builtin_amdgcn_permlane32_swap(y, y, false, false);
        const bool hi = __lane_id() & 32;
        a = hi ? rx[0] : rx[1];
        b = hi ? ry[0] : ry[1];
    }
}
template <int STEP = 0>
__device__ __forceinline__ unsigned long long wave_max_key_from(uint32_t hi, uint32_t lo) {
    if constexpr (STEP == 6) {
        return ((unsigned long long)hi << 32) | lo;
    } else {
        uint32_t ph, pl;
        partner<STEP>(ph, pl, hi, lo);
        const bool take = ph > hi || (ph == hi && pl > lo);
        return wave_max_key_from<STEP + 1>(take ? ph : hi, take ? pl : lo);
    }
}
__device__ __forceinline__ unsigned long long wave_max_key(unsigned long long x) {
    return wave_max_key_from<0>((uint32_t)(x >> 32), (uint32_t)x);
}
template <int STEP = 0>
__device__ __forceinline__ float wave_max_f(float x) {
    if constexpr (STEP == 6) {
        return x;
    } else {
        uint32_t p, unused;
        partner<STEP>(p, unused, __float_as_uint(x), 0u);
        return wave_max_f<STEP + 1>(fmaxf(x, __uint_as_float(p)));
    }
}
template <int STEP = 0>
__device__ __forceinline__ float wave_sum_f(float x) {
    if constexpr (STEP == 6) {
        return x;
    } else {
        uint32_t p, unused;
        partner<STEP>(p, unused, __float_as_uint(x), 0u);
        // the pair is added in lane order, so both lanes get the same bits
        const float o = __uint_as_float(p);
        const bool low = STEP < 4 ? true : !(__lane_id() & (STEP == 4 ? 16 : 32));
        return wave_sum_f<STEP + 1>(low ? x + o : o + x);
    }
}

template <int STEP = 0>
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
    if constexpr (STEP == 6) {
        return x;
    } else {
        uint32_t p, unused;
        partner<STEP>(p, unused, x, 0u);
        return wave_or<STEP + 1>(x | p);
    }
}

// Tag of the record words of a call, in their high 32 bits: the host's epoch
// in [1, 2^31), or, for a call captured into a graph (epoch 0), the source's
// counter in the workspace with bit 31 set, which the source's merger
// advances once it has every record.  c0 receives the counter value.
__device__ __forceinline__ unsigned long long call_tag(unsigned long long epoch, const unsigned long long *ctr,
                                                       unsigned long long &c0) {
    if (epoch != 0) return (epoch & 0xffffffffull) << 32;
    c0 = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return (0x80000000ull | ((c0 % 0x7fffffffull) + 1)) << 32;
}

__device__ __forceinline__ void store_word(unsigned long long *p, unsigned long long tag, uint32_t v) {
    __hip_atomic_store(p, tag | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Raw buffer resource over the first `bytes` bytes at p: loads past the end
// return 0 without a memory access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *p, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, 0x00020000);
}
// 4-byte buffer load at voff + soff; aux 2 = non-temporal.
__device__ __forceinline__ uint32_t buf_load(__amdgpu_buffer_rsrc_t r, int voff, int soff, int aux) {
    return aux ? __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 2)
               : __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}

// Record of one (row, slice): m, s, then c values and c token ids; every
// word is (call tag << 32 | 32-bit payload).
__host__ __device__ constexpr int rec_words(int c) { return 2 + 2 * c; }

// The c best of n keys in LDS, by rank: thread e counts the keys above key
// e, and a key of rank < c goes to out[rank] (keys other than 0 are
// distinct, so the ranks are).  keys is 16-byte aligned and, for odd n,
// keys[n] is 0 (a 0 key is above none); out[0..c) must hold 0 beforehand.
// The keys are read two at a time, eight reads in flight.
__device__ __forceinline__ void rank_top_keys(const unsigned long long *keys, int n, int c,
                                              unsigned long long *out) {
    const ulonglong2 *k2 = reinterpret_cast<const ulonglong2 *>(keys);
    const int n2 = (n + 1) / 2;
    for (int e = threadIdx.x; e < n; e += kThreads) {
        const unsigned long long ke = keys[e];
        int rank = 0;
        int j = 0;
        for (; j + 8 <= n2; j += 8) {
            ulonglong2 q[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) q[u] = k2[j + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) rank += (q[u].x > ke) + (q[u].y > ke);
        }
        for (; j < n2; ++j) {
            const ulonglong2 q = k2[j];
            rank += (q.x > ke) + (q.y > ke);
        }
        if (rank < c && ke != 0ull) out[rank] = ke;
    }
}

// Barrier for LDS only: waits for this wave's LDS operations, not for its
// global loads still in flight (unlike __syncthreads).
__device__ __forceinline__ void lds_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt left open
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Maximum over each block of kWaves adjacent lanes (the first log2(kWaves)
// butterfly steps); every lane of a block ends with its block's maximum.
template <int STEP = 0>
__device__ __forceinline__ float block_max(float x) {
    if constexpr ((1 << STEP) >= kWaves) {
        return x;
    } else {
        uint32_t p, unused;
        partner<STEP>(p, unused, __float_as_uint(x), 0u);
        return block_max<STEP + 1>(fmaxf(x, __uint_as_float(p)));
    }
}

// LDS of a slice workgroup and of a merger; a workgroup is one or the
// other, so the kernel holds them in one union.
struct SliceLds {
    alignas(16) unsigned long long comp[kCap + 2 + kWave];  // candidate keys, then one spare slot per lane
    alignas(16) unsigned long long bkey[kWave];     // the 64 block maxima as keys
    unsigned long long best[16];
    unsigned long long xwin[kWaves];                // exact path: each wave's best key of a round
    uint32_t ban_bits[kSliceMax / 32];
    int nban[kWaves];                               // banned positions held by each wave
    int ncand;
    float wm[kWaves], ws[kWaves];
};
struct MergeLds {
    alignas(16) unsigned long long keys[kMergeCap + 2];
    alignas(16) unsigned long long surv[kMergeCap + 2];
    unsigned long long best[16];
    unsigned long long hc;
    uint32_t w32[kMergeWords];
    float bsc[16];
    int stale, nsurv;
};
union SelectLds {
    SliceLds slice;
    MergeLds merge;
};

// Slice workgroup: row r, vocabulary [v0, v1), len = v1 - v0 positions.
// The workgroup reads the 16-byte-aligned window that starts a = (address of
// logit v0 / 4) mod 4 positions before v0, so every load is 16 bytes whatever
// V and the slice bounds are; window position w is slice position w - a.
// Value j of a thread sits at window position lbase + offs(j), lbase = 4 *
// thread: load g of the workgroup covers window positions [1024g, 1024g + 1024).
// Every 16-byte chunk the window reads holds at least one logit of the slice,
// so no read leaves the pages of the logits.
__device__ __forceinline__ constexpr int offs(int j) { return (j / 4) * kThreads * 4 + j % 4; }

__device__ void select_slice(SliceLds &L, const float *__restrict__ logits, const int32_t *__restrict__ tokens,
                             int ld, int t, int n, unsigned long long *__restrict__ part, int r, int s, int V, int c,
                             int NS, int SL, unsigned long long tag)
{
    constexpr int kGroups = kPer / 4;          // 16-byte loads per thread
    constexpr int kSpan = kThreads * 4;        // window positions per load
    constexpr float kLog2e = 1.4426950408889634f;
    uint32_t *ban_bits = L.ban_bits;
    int *nban = L.nban;
    unsigned long long *comp = L.comp, *best = L.best, *bkey = L.bkey, *xwin = L.xwin;
    float *wm = L.wm, *ws = L.ws;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
    // trace words: 0 start, 1 data in, 2 threshold, 3 collected, 4 end,
    // 5 hardware ids, 6 candidates, 7 = 0 (a slice)
    unsigned long long *trs = trace_slot();
    trace::stamp(trs, 0);
    const int v0 = s * SL, v1 = min(V, v0 + SL), len = max(0, v1 - v0);
    const float *x = logits + (size_t)r * V + v0;
    const int a = (int)((reinterpret_cast<uintptr_t>(x) >> 2) & 3);
    const int wl = len > 0 ? a + len : 0;                 // window length (an empty slice reads nothing)
    const int ng = (wl + kSpan - 1) / kSpan;              // loads holding any slice position
    const int nfull = wl / kSpan;                         // loads [a ? 1 : 0, nfull) hold only slice positions
    const int lbase = tid * 4;

    // This thread's first window of the history (positions tid .. tid+n-1)
    // and the row's suffix, loaded before the logits: loads complete in
    // order, so the ban scan can start without waiting for the slice.  All
    // are unconditional buffer loads (reads past the range return 0), so no
    // branch separates them and each use waits only for its own loads.
    const bool bans = n >= 1 && t >= n;
    const int32_t *h = bans ? tokens + (size_t)r * ld : tokens;
    const auto tres = buf_rsrc(h, bans ? t * 4 : 0);
    const bool win0 = bans && n <= kNMax && tid <= t - n;
    int32_t hw[kNMax], sf[kNMax - 1];
#pragma unroll
    for (int q = 0; q < kNMax; ++q) hw[q] = (int32_t)buf_load(tres, (tid + q) * 4, 0, 0);
#pragma unroll
    for (int q = 0; q < kNMax - 1; ++q) sf[q] = (int32_t)buf_load(tres, (t - n + 1 + q) * 4, 0, 0);
    float val[kPer];
    {
        const auto res = buf_rsrc(x - a, wl * 4);
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const u32x4_t q = __builtin_bit_cast(
                u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(res, lbase * 4, g * kSpan * 4, 2));
#pragma unroll
            for (int e = 0; e < 4; ++e) val[4 * g + e] = __uint_as_float(q[e]);
        }
    }

    // banned tokens of this slice (Algorithm 1), while the loads are in
    // flight, as bits of window positions: a thread's 4 values share a word
    for (int i = tid; i < (wl + 31) / 32; i += kThreads) ban_bits[i] = 0u;
    if (tid < 16) best[tid] = 0ull;
    if (tid < kWaves) nban[tid] = 0;
    if (tid == 0) L.ncand = 0;
    lds_barrier();
    if (bans) {
        const int suffix = t - n + 1;
        auto ban = [&](int32_t v) {
            if (v >= v0 && v < v1) {
                const int w = v - v0 + a;
                atomicOr(&ban_bits[w >> 5], 1u << (w & 31));
                atomicAdd(&nban[(w % kSpan) / (4 * kWave)], 1);   // the wave whose lanes hold w
            }
        };
        if (win0) {
            // the first window, already in registers; the suffix is wave-uniform
            int diff = 0;
#pragma unroll
            for (int q = 0; q < kNMax - 1; ++q)
                if (q < n - 1) diff |= hw[q] ^ sf[q];
            int32_t v = 0;
#pragma unroll
            for (int q = 0; q < kNMax; ++q) v = q == n - 1 ? hw[q] : v;
            if (diff == 0) ban(v);
        }
        // the remaining windows (long histories, or n > kNMax), from memory
        for (int j = n <= kNMax ? tid + kThreads : tid; j <= t - n; j += kThreads) {
            int diff = 0;  // no early exit: the window's loads go out together
            for (int q = 0; q < n - 1; ++q) diff |= h[j + q] ^ h[suffix + q];
            if (diff == 0) ban(h[j + n - 1]);
        }
    }
    lds_barrier();

    // the lane's maximum over its positions, load by load as they arrive;
    // window positions outside the slice become -inf
    float m = -INFINITY;
    float gm[kGroups];   // maximum of each load's four values
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        gm[g] = -INFINITY;
        if (g < ng) {
            if (g >= nfull || (g == 0 && a != 0)) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    val[4 * g + e] = (unsigned)(lbase + offs(4 * g + e) - a) < (unsigned)len ? val[4 * g + e]
                                                                                          : -INFINITY;
            }
            gm[g] = fmaxf(fmaxf(val[4 * g], val[4 * g + 1]), fmaxf(val[4 * g + 2], val[4 * g + 3]));
            m = fmaxf(m, gm[g]);
        }
    }
    // the wave's (max, sum of exp) over every logit, banned or not
    const float mw = wave_max_f(m);
    if (trs) {
        asm volatile("" ::"v"(mw));   // the stamp after the data
        trace::stamp(trs, 1);
    }
    float sum = 0.f;
    if (mw != -INFINITY) {
        const float sh = mw * kLog2e;
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            if (g < ng)
#pragma unroll
                for (int e = 0; e < 4; ++e) sum += __builtin_amdgcn_exp2f(fmaf(val[4 * g + e], kLog2e, -sh));
    }
    const float sw = wave_sum_f(sum);

    // Banned positions cannot be candidates: with any ban in the slice, every
    // wave turns its banned values into -inf (after the sums, which take
    // every token) and retakes its load maxima.
    int nb = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) nb += nban[w];
    nb = __builtin_amdgcn_readfirstlane(nb);
    float cm = m;
    if (nb > 0) {
        cm = -INFINITY;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            if (g < ng) {
                const uint32_t bits = ban_bits[(lbase + g * kSpan) >> 5] >> ((lbase + g * kSpan) & 31);
#pragma unroll
                for (int e = 0; e < 4; ++e) val[4 * g + e] = ((bits >> e) & 1u) ? -INFINITY : val[4 * g + e];
                gm[g] = fmaxf(fmaxf(val[4 * g], val[4 * g + 1]), fmaxf(val[4 * g + 2], val[4 * g + 3]));
                cm = fmaxf(cm, gm[g]);
            }
        }
    }
    // Threshold tau: the c-th largest of the slice's 64 block maxima (blocks
    // of kWaves adjacent lanes of one wave, so kBlocks per wave).  The c
    // largest blocks each hold a distinct unbanned position at or above tau,
    // so the slice's c best candidates all lie at or above it.  Each lane
    // ranks one block maximum (as a key with its block index, so the 64 keys
    // are distinct) against all 64; every wave finds the same tau.
    const float bm = block_max(cm);
    const int bidx = wv * kBlocks + lane / kWaves;
    if ((lane & (kWaves - 1)) == 0) bkey[bidx] = ((unsigned long long)ordered(bm) << 32) | (uint32_t)~bidx;
    if (lane == 0) {
        wm[wv] = mw;
        ws[wv] = sw;
    }
    lds_barrier();
    float tau;
    {
        const unsigned long long mine = bkey[lane];
        const ulonglong2 *b2 = reinterpret_cast<const ulonglong2 *>(bkey);
        // four reads in flight at a time
        int rank = 0;
#pragma unroll
        for (int q0 = 0; q0 < kWave / 2; q0 += 4) {
            ulonglong2 o[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) o[u] = b2[q0 + u];
#pragma unroll
            for (int u = 0; u < 4; ++u) rank += (o[u].x > mine) + (o[u].y > mine);
        }
        const unsigned long long at = __builtin_amdgcn_ballot_w64(rank == c - 1);
        const int src = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(at));   // one lane: the keys are distinct
        tau = unordered((uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(mine >> 32), src));
    }
    if (trs) {
        asm volatile("" ::"v"(tau));
        trace::stamp(trs, 2);
    }

    // Collect the positions at or above tau as keys.  Positions outside the
    // slice hold -inf, below a finite tau; for tau = -inf they become NaN
    // first, which compares false.  A banned position holds -inf, so it is a
    // -inf candidate.  Each lane takes its places with one LDS atomic; a
    // value below tau is written to the lane's spare slot instead, so the
    // stores need no branch.
    if (tau == -INFINITY) {
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            if (g < ng && (g >= nfull || (g == 0 && a != 0)))
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    val[4 * g + e] = (unsigned)(lbase + offs(4 * g + e) - a) < (unsigned)len ? val[4 * g + e] : NAN;
    }
    uint32_t lhot = 0u;   // this lane's loads holding a value at or above tau
#pragma unroll
    for (int g = 0; g < kGroups; ++g) lhot |= (g < ng && gm[g] >= tau) ? 1u << g : 0u;
    const uint32_t hot = __builtin_amdgcn_readfirstlane(wave_or(lhot));
    int nh = 0;
#pragma unroll
    for (int g = 0; g < kGroups; ++g)
        if ((hot >> g) & 1u)
#pragma unroll
            for (int e = 0; e < 4; ++e) nh += val[4 * g + e] >= tau;
    int at = 0;
    if (nh > 0) at = atomicAdd(&L.ncand, nh);
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        if ((hot >> g) & 1u) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int j = 4 * g + e;
                const bool ok = val[j] >= tau && at < kCap;
                comp[ok ? at : kCap + 2 + lane] = make_key(val[j], (uint32_t)(v0 + lbase + offs(j) - a));
                at += ok;
            }
        }
    }
    lds_barrier();
    const int total = L.ncand;
    trace::stamp(trs, 3);
    trace::put(trs, 6, (unsigned long long)total);
    unsigned long long *rec = part + ((size_t)r * NS + s) * rec_words(c);
    if (total <= kWave) {
        // Few candidates: wave 0 ranks them in registers and writes the
        // record; the other waves are done.
        if (wv != 0) return;
        const unsigned long long ke = lane < total ? comp[lane] : 0ull;
        const ulonglong2 *k2 = reinterpret_cast<const ulonglong2 *>(comp);
        int rank = 0;
        for (int q = 0; q < (total + 1) / 2; ++q) {
            const ulonglong2 o = k2[q];
            rank += (o.x > ke) + (q * 2 + 1 < total && o.y > ke);
        }
        if (lane < total && rank < c) {
            store_word(rec + 2 + rank, tag, __float_as_uint(unordered((uint32_t)(ke >> 32))));
            store_word(rec + 2 + c + rank, tag, ~(uint32_t)ke);
        }
        // an empty slot (fewer positions than c) is a -inf value at index ~0
        if (lane >= total && lane < c) {
            store_word(rec + 2 + lane, tag, __float_as_uint(-INFINITY));
            store_word(rec + 2 + c + lane, tag, 0xffffffffu);
        }
    } else {
        if (total <= kCap) {
            // the keys ranked among themselves by every thread
            if (tid == 0) {
                comp[total] = 0ull;
                comp[total + 1] = 0ull;
            }
            if (tid < 16) best[tid] = 0ull;
            lds_barrier();
            rank_top_keys(comp, total, c, best);
        } else {
            // Exact path (more than kCap values at the threshold, e.g. equal
            // logits): c rounds, each taking the best key below the last one.
            // The values become their order-preserving bits in place (0
            // outside the slice, below every position's) and the index half of
            // a key is formed in each round, so no 64-bit key array stays live
            // across the rounds.
#pragma unroll
            for (int g = 0; g < kGroups; ++g) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int j = 4 * g + e;
                    const bool in = (unsigned)(lbase + offs(j) - a) < (unsigned)len;
                    val[j] = __uint_as_float(in ? ordered(val[j]) : 0u);
                }
            }
            uint32_t last_hi = ~0u, last_lo = ~0u;
            for (int q = 0; q < c; ++q) {
                // ~index of offset 0 (~(i + d) = ~i - d), opaque to the compiler in
                // each round so that the 64 index halves are not kept across rounds
                uint32_t lo0 = ~(uint32_t)(v0 + lbase - a);
                asm volatile("" : "+v"(lo0));
                // (bh, bl) starts below every key whose high half is not 0, and
                // positions outside the slice (high half 0) never rise above it
                uint32_t bh = 0u, bl = ~0u;
#pragma unroll
                for (int j = 0; j < kPer; ++j) {
                    const uint32_t hi = __float_as_uint(val[j]);
                    const uint32_t lo = lo0 - (uint32_t)offs(j);
                    const bool below = hi < last_hi || (hi == last_hi && lo < last_lo);
                    const bool above = hi > bh || (hi == bh && lo > bl);
                    bh = below && above ? hi : bh;
                    bl = below && above ? lo : bl;
                }
                const unsigned long long b = wave_max_key(bh ? ((unsigned long long)bh << 32) | bl : 0ull);
                __syncthreads();  // the previous round's reads of xwin are done
                if (lane == 0) xwin[wv] = b;
                __syncthreads();
                unsigned long long wmax = xwin[0];
#pragma unroll
                for (int w = 1; w < kWaves; ++w) wmax = xwin[w] > wmax ? xwin[w] : wmax;
                if (tid == 0) best[q] = wmax;
                last_hi = (uint32_t)(wmax >> 32);
                last_lo = (uint32_t)wmax;
            }
        }
        lds_barrier();
        if (tid < c) {
            const unsigned long long kk = best[tid];
            // an empty key (fewer positions than c) is a -inf value at index ~0
            store_word(rec + 2 + tid, tag, kk ? __float_as_uint(unordered((uint32_t)(kk >> 32)))
                                              : __float_as_uint(-INFINITY));
            store_word(rec + 2 + c + tid, tag, kk ? ~(uint32_t)kk : 0xffffffffu);
        }
    }
    // the slice's (max, sum of exp): the waves' sums rescaled to the slice maximum
    if (tid == 0) {
        float M = wm[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) M = fmaxf(M, wm[w]);
        float S = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w)
            S += wm[w] == -INFINITY ? 0.f : ws[w] * __builtin_amdgcn_exp2f((wm[w] - M) * kLog2e);
        store_word(rec, tag, __float_as_uint(M));
        store_word(rec + 1, tag, __float_as_uint(S));
    }
    trace::stamp(trs, 4);
    trace::put(trs, 5, trace::where());
    trace::put(trs, 7, 0);
}

// Merger of source b: reads the k * NS records of its rows into LDS (every
// word at once, re-reading only words that do not carry this call's tag yet),
// then ranks.
__device__ void select_merge(MergeLds &L, const float *__restrict__ beam_scores,
                             const unsigned long long *__restrict__ part, float *__restrict__ out_scores,
                             int32_t *__restrict__ out_beam, int32_t *__restrict__ out_token, int b, int k, int V,
                             int c, int NS, unsigned long long tag)
{
    uint32_t *w32 = L.w32;
    float *bsc = L.bsc;
    unsigned long long *keys = L.keys, *surv = L.surv, *best = L.best;
    int &stale = L.stale;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int W = rec_words(c);
    const int nw = k * NS * W;
    const unsigned long long *recs = part + (size_t)b * k * NS * W;
    // trace words: 0 start, 1 records in, 4 end, 5 hardware ids,
    // 6 survivors, 7 = 1 (a merger)
    unsigned long long *trs = trace_slot();
    trace::stamp(trs, 0);
    if (tid == 0) {
        stale = 0;
        L.nsurv = 0;
        L.hc = 0ull;
    }
    if (tid < 16) best[tid] = 0ull;
    if (tid < k) bsc[tid] = beam_scores[(size_t)b * k + tid];
    // the survivors' array holds 0 past its last entry (a 0 key ranks below
    // every other), so no entry needs clearing after the packing
    for (int e = tid; e < kMergeCap + 2; e += kThreads) surv[e] = 0ull;
    constexpr int kPerThread = kMergeWords / kThreads;
    unsigned long long wv[kPerThread];
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
        const int e = tid + q * kThreads;
        wv[q] = e < nw ? __hip_atomic_load(recs + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : tag;
    }
    // re-read every word still without the tag together, so the wait ends
    // one round trip after the last record lands
    constexpr unsigned long long kHi = 0xffffffff00000000ull;
    for (int spin = 0; spin < kMaxSpins; ++spin) {
        bool pending = false;
#pragma unroll
        for (int q = 0; q < kPerThread; ++q) pending |= (wv[q] & kHi) != tag;
        if (!pending) break;
        __builtin_amdgcn_s_sleep(2);
#pragma unroll
        for (int q = 0; q < kPerThread; ++q)
            if ((wv[q] & kHi) != tag)
                wv[q] = __hip_atomic_load(recs + tid + q * kThreads, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    bool old = false;
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
        const int e = tid + q * kThreads;
        old |= (wv[q] & kHi) != tag;
        if (e < nw) w32[e] = (uint32_t)wv[q];
    }
    __syncthreads();
    trace::stamp(trs, 1);
    if (old) stale = 1;
    // Every slice candidate, scored; each thread takes its row's lse from the
    // row's slice records (the maximum, then the rescaled sums in slice
    // order).  Keys are stored position-major, key (j, record q) at
    // j * nrec + q, so the records' heads (j = 0) are the first nrec keys.
    const int ncand = k * NS * c;
    const int nrec = k * NS;
    constexpr float kL2e = 1.4426950408889634f;
    for (int e = tid; e < ncand; e += kThreads) {
        const int i = e / (NS * c), rem = e - i * NS * c, s = rem / c, j = rem - s * c;
        const uint32_t *rw = w32 + i * NS * W;
        float M = -INFINITY;
        for (int u = 0; u < NS; ++u) M = fmaxf(M, __uint_as_float(rw[u * W]));
        float S = 0.f;
        for (int u = 0; u < NS; ++u) {
            const float ms = __uint_as_float(rw[u * W]);
            const float ss = __uint_as_float(rw[u * W + 1]);
            S += ms == -INFINITY ? 0.f : ss * __builtin_amdgcn_exp2f((ms - M) * kL2e);
        }
        const float lr = M == -INFINITY ? -INFINITY : M + logf(S);
        const float x = __uint_as_float(rw[s * W + 2 + j]);
        const uint32_t v = rw[s * W + 2 + c + j];
        const float sc = (lr == -INFINITY || x == -INFINITY) ? -INFINITY : bsc[i] + (x - lr);
        // an empty slot (v = ~0) ranks below every candidate
        keys[j * nrec + i * NS + s] = v == 0xffffffffu ? 0ull : make_key(sc, (uint32_t)i * (uint32_t)V + v);
    }
    __syncthreads();
    // Prune: the heads (first candidates) of the k * NS records are distinct
    // candidates, so no candidate below the c-th largest head is among the c
    // best.  The heads are ranked among themselves, the candidates at or
    // above that head are packed, and only they are ranked.
    if (nrec >= c) {
        const ulonglong2 *h2 = reinterpret_cast<const ulonglong2 *>(keys);
        for (int q = tid; q < nrec; q += kThreads) {
            const unsigned long long hq = keys[q];
            int rank = 0;
            int q2 = 0;
            for (; 2 * q2 + 1 < nrec; ++q2) {
                const ulonglong2 o = h2[q2];
                rank += (o.x > hq) + (o.y > hq);
            }
            if (2 * q2 < nrec) rank += keys[2 * q2] > hq;
            if (rank == c - 1) L.hc = hq;   // heads other than 0 are distinct
        }
        __syncthreads();
    }
    const unsigned long long hc = L.hc;
    for (int e0 = 0; e0 < ncand; e0 += kThreads) {
        const int e = e0 + tid;
        const unsigned long long ke = e < ncand ? keys[e] : 0ull;
        const bool keep = ke != 0ull && ke >= hc;
        const unsigned long long m = __builtin_amdgcn_ballot_w64(keep);
        int base = 0;
        if (m != 0ull && lane == 0) base = atomicAdd(&L.nsurv, (int)__popcll(m));
        base = __builtin_amdgcn_readfirstlane(base);
        if (keep)
            surv[base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u))] = ke;
    }
    __syncthreads();
    const int ns = L.nsurv;
    rank_top_keys(surv, ns, c, best);
    __syncthreads();
    if (tid < c) {
        const unsigned long long kk = best[tid];
        const uint32_t f = ~(uint32_t)kk;
        const bool bad = stale || kk == 0ull;
        out_scores[(size_t)b * c + tid] = bad ? NAN : unordered((uint32_t)(kk >> 32));
        out_beam[(size_t)b * c + tid] = bad ? -1 : (int32_t)(f / (uint32_t)V);
        out_token[(size_t)b * c + tid] = bad ? -1 : (int32_t)(f % (uint32_t)V);
    }
    trace::stamp(trs, 4);
    trace::put(trs, 5, trace::where());
    trace::put(trs, 6, (unsigned long long)ns);
    trace::put(trs, 7, 1);
}

__global__ __launch_bounds__(kThreads) void beam_select_kernel(
    const float *__restrict__ logits, const float *__restrict__ beam_scores, const int32_t *__restrict__ tokens,
    int ld, int t, int n, float *__restrict__ out_scores, int32_t *__restrict__ out_beam,
    int32_t *__restrict__ out_token, unsigned long long *__restrict__ part, int rows, int k, int V, int c,
    int NS, int SL, unsigned long long epoch, unsigned long long *__restrict__ ctr)
{
    __shared__ SelectLds lds;
    const int g = blockIdx.x;
    const int b = g < rows * NS ? g / NS / k : g - rows * NS;
    unsigned long long c0 = 0;
    const unsigned long long tag = call_tag(epoch, ctr + b, c0);
    if (g < rows * NS) {
        select_slice(lds.slice, logits, tokens, ld, t, n, part, g / NS, g % NS, V, c, NS, SL, tag);
    } else {
        select_merge(lds.merge, beam_scores, part, out_scores, out_beam, out_token, b, k, V, c, NS, tag);
        // a captured call: the merger has every record (or its wait ran
        // out), so every slice of the source has read the counter; the next
        // call takes the next value (skipping one after a wait that ran out,
        // so that a late record of this call never passes for the next's)
        if (epoch == 0 && threadIdx.x == 0)
            __hip_atomic_store(ctr + b, c0 + (lds.merge.stale ? 2 : 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace

namespace {
std::atomic<int> g_slices_override{0};
}  // namespace

hipError_t set_select_trace(unsigned long long *buf, unsigned int cap) {
#if FS_TRACE
    const trace::Target t{buf, cap};
    return hipMemcpyToSymbol(HIP_SYMBOL(g_trace), &t, sizeof(t));
#else
    (void)buf;
    (void)cap;
    return hipErrorNotSupported;
#endif
}

int set_select_slices_override(int slices) {
    return g_slices_override.exchange(slices > 0 ? slices : 0, std::memory_order_relaxed);
}

int beam_select_slices(int rows, int V, int k, int c) {
    // About kTargetWorkgroups slice workgroups, slices of at least 1024
    // logits, and no more than one merger ranks; a slice's window (slice plus
    // up to 3 leading positions) fits the kSliceMax positions of a workgroup.
    // set_select_slices_override sets the count within the same limits.
    constexpr int kTargetWorkgroups = 512;
    const int by_size = (V + kSliceMax - 4) / (kSliceMax - 3);
    const int by_cand = kMergeCap / (k * c > 0 ? k * c : 1);
    const int by_words = kMergeWords / (k * rec_words(c) > 0 ? k * rec_words(c) : 1);
    const int forced = g_slices_override.load(std::memory_order_relaxed);
    int ns = forced > 0 ? forced : (kTargetWorkgroups + rows - 1) / (rows > 0 ? rows : 1);
    if (forced <= 0) ns = ns < (V + 1023) / 1024 ? ns : (V + 1023) / 1024;
    ns = ns < by_cand ? ns : by_cand;
    ns = ns < by_words ? ns : by_words;
    ns = ns < V ? ns : V;
    return ns > by_size ? ns : (by_size > 0 ? by_size : 1);
}

int beam_select_max_candidates() { return kMergeCap; }
int beam_select_max_record_words() { return kMergeWords; }

size_t beam_select_workspace_words(int B, int k, int V, int c) {
    const int NS = beam_select_slices(B * k, V, k, c);
    return (size_t)B * k * NS * rec_words(c) + B;   // the records, then one counter per source
}

hipError_t launch_beam_select(const float *logits, const float *beam_scores, const int32_t *tokens, int ld,
                              int t, int n, float *out_scores, int32_t *out_beam, int32_t *out_token, int B,
                              int k, int V, int c, unsigned long long *workspace, unsigned long long epoch,
                              hipStream_t stream)
{
    const int rows = B * k;
    const int NS = beam_select_slices(rows, V, k, c);
    const int SL = (V + NS - 1) / NS;
    const long long nblk = (long long)rows * NS + B;
    unsigned long long *ctr = workspace + (size_t)rows * NS * rec_words(c);
    hipLaunchKernelGGL(beam_select_kernel, dim3((unsigned)nblk), dim3(kThreads), 0, stream, logits, beam_scores,
                       tokens, ld, t, n, out_scores, out_beam, out_token, workspace, rows, k, V, c, NS, SL, epoch,
                       ctr);
    return hipGetLastError();
}

}  // namespace fs
