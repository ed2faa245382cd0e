// Encoder-decoder cross-attention over a de-duplicated K/V cache, for gfx950.
//
// The operation is Eq. 4 of the paper (Appendix B): the k beam queries of
// source b read the one copy K[b], V[b] of that source's encoder keys and
// values, and each computes softmax(q K^T / sqrt(D)) V over the valid keys
// j < src_len[b].  Per head it is a GEMV-like contraction with k query rows
// (about k flop per byte of K/V), so it is bound by HBM bandwidth.  The
// kernel reads every valid K/V byte exactly once with coalesced,
// non-temporal 16-byte loads and keeps all k beams' work on that data in
// registers.
//
// One launch, split-KV:
//   One workgroup per (source b, head h, chunk c of C keys); 4 waves, each
//   owning one tile of the chunk.  In a tile a group of kLpr lanes shares one
//   row (16 bytes per lane), so a wave instruction reads kRpi whole rows.
//     QK^T:  each lane dots its 16 bytes of the row with the same 16 bytes of
//            every beam's query (held in registers); a butterfly inside the
//            lane group completes the k scores.
//     softmax: tile maximum and sum per beam by cross-group butterflies; the
//            running (max, sum) of the online softmax is wave-uniform.
//     PV:    the same lane layout reads V; each lane accumulates k x (its 16
//            bytes of dims) in fp32.
//   The waves' states are merged through LDS in a fixed order.  A source
//   whose valid keys fit in one chunk is finished there.  Otherwise each
//   chunk stores its partial (max, sum, unnormalised output) in the
//   workspace and exits without waiting.
//   One merger workgroup per (b, h), placed after all chunk workgroups in
//   the grid (so dispatched after them), reads the chunks' records, merges
//   them in chunk order, normalises and writes the output.  Each record word
//   carries a tag of the call, so the merger knows when a record is
//   complete; no fence or clearing of the workspace is needed.  The tag is
//   the host's call epoch, or, for a call captured into a graph, a per-row
//   counter in the workspace that the row's merger advances.
// Rows j >= src_len[b] are never read.  The chunk size depends only on the
// row size, and each beam's arithmetic is the same whatever k is, so the
// output bits do not depend on k, B or the beam's position.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "launch.h"
#include "ngram_row.h"
#include "trace.h"

namespace fs {
namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWave * kWaves;
constexpr int kIt = 8;   // row loads of K (and of V) per lane per tile
constexpr int kXcds = 8; // MI355X: workgroups go round-robin to 8 XCDs
constexpr int kCus = 256;                // MI355X compute units
constexpr int kWhole2MinRows = 128;      // fewer (b, h) rows than this are split across workgroups

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <bool BF16>
struct Elem {
    static constexpr int size = BF16 ? 2 : 4;
    static constexpr int per16 = 16 / size;  // elements in 16 bytes
};

template <int D, bool BF16>
struct Geo {
    static constexpr int kEpl = Elem<BF16>::per16;   // elements per lane slice
    static constexpr int kLpr = D / kEpl;            // lanes sharing one row
    static constexpr int kRpi = kWave / kLpr;        // rows per wave instruction
    static constexpr int kTile = kIt * kRpi;         // keys per wave tile
    static constexpr int kChunk = kWaves * kTile;    // keys per workgroup
    static constexpr int kDup = kLpr > kIt ? kLpr / kIt : 1;   // lanes sharing a score row
    static constexpr int kRows = kLpr < kIt ? kIt / kLpr : 1;  // score rows per lane
    static constexpr int kPStride = kTile + kTile / 8;     // LDS rows per wave (padded)
    static_assert(kLpr >= 2 && kLpr <= 32, "row must be 32..512 bytes");
    static_assert(kIt == 8 || kIt == 16, "the row-load count must be a power of two >= 8");
};

__device__ __forceinline__ uint4 load_nt(const uint4 *p) {
    const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(t.x, t.y, t.z, t.w);
}

// Buffer resource over the first `bytes` bytes at p (raw addressing, no
// stride): loads past the end return zero without touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void *p, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, 0x00020000);
}
// 16-byte non-temporal buffer load at byte offset voff + soff.
__device__ __forceinline__ uint4 load_rows(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const u32x4_t t = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 2));
    return make_uint4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Dot product of two 16-byte slices, accumulated into c in element order.
template <bool BF16>
__device__ __forceinline__ float dot16(uint4 a, uint4 b, float c) {
    if constexpr (BF16) {
        c = dot2_bf16(a.x, b.x, c);
        c = dot2_bf16(a.y, b.y, c);
        c = dot2_bf16(a.z, b.z, c);
        c = dot2_bf16(a.w, b.w, c);
    } else {
        c = fmaf(__uint_as_float(a.x), __uint_as_float(b.x), c);
        c = fmaf(__uint_as_float(a.y), __uint_as_float(b.y), c);
        c = fmaf(__uint_as_float(a.z), __uint_as_float(b.z), c);
        c = fmaf(__uint_as_float(a.w), __uint_as_float(b.w), c);
    }
    return c;
}

// Unpack a 16-byte slice to fp32 values (exact).
template <bool BF16>
__device__ __forceinline__ void unpack16(uint4 a, float *f) {
    if constexpr (BF16) {
        f[0] = bf16_lo(a.x); f[1] = bf16_hi(a.x);
        f[2] = bf16_lo(a.y); f[3] = bf16_hi(a.y);
        f[4] = bf16_lo(a.z); f[5] = bf16_hi(a.z);
        f[6] = bf16_lo(a.w); f[7] = bf16_hi(a.w);
    } else {
        f[0] = __uint_as_float(a.x); f[1] = __uint_as_float(a.y);
        f[2] = __uint_as_float(a.z); f[3] = __uint_as_float(a.w);
    }
}

// ---- cross-lane exchange ---------------------------------------------------
// DPP stays inside a row of 16 lanes, ds_swizzle inside 32 lanes, and
// ds_bpermute covers the whole wave.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}
template <int PATTERN>
__device__ __forceinline__ float swizzle(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), PATTERN));
}
__device__ __forceinline__ float lane_xor(float x, int mask) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((__lane_id() ^ mask) << 2,
                                                                  __builtin_bit_cast(int, x)));
}

// Value of lane (lane ^ MASK), for MASK a power of two below 64.
template <int MASK>
__device__ __forceinline__ float xor_lane(float x) {
    if constexpr (MASK == 1) return dpp<0xB1>(x);              // quad_perm [1,0,3,2]
    else if constexpr (MASK == 2) return dpp<0x4E>(x);         // quad_perm [2,3,0,1]
    else if constexpr (MASK == 8) return dpp<0x128>(x);        // row_ror:8 == xor 8 in a row
    else if constexpr (MASK < 32) return swizzle<0x1F | (MASK << 10)>(x);  // bit mode, xor MASK
    else return lane_xor(x, MASK);
}

// Sum over the kLpr lanes of a row group (every lane of the group gets the
// bit-identical result: each step pairs lanes and adds commutatively).
template <int G>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (G >= 2) x += dpp<0xB1>(x);
    if constexpr (G >= 4) x += dpp<0x4E>(x);
    if constexpr (G >= 8) x += dpp<0x141>(x);   // row_half_mirror: other quad of the 8
    if constexpr (G >= 16) x += dpp<0x140>(x);  // row_mirror: other 8 of the 16
    if constexpr (G >= 32) x += swizzle<0x401F>(x);
    return x;
}

// Reduction over the row groups of a wave (lanes sharing lane % G).
template <int G, int MASK = G>
__device__ __forceinline__ float groups_max(float x) {
    if constexpr (MASK < kWave) {
        x = fmaxf(x, xor_lane<MASK>(x));
        return groups_max<G, MASK * 2>(x);
    } else {
        return x;
    }
}
template <int G, int MASK = G>
__device__ __forceinline__ float groups_sum(float x) {
    if constexpr (MASK < kWave) {
        x += xor_lane<MASK>(x);
        return groups_sum<G, MASK * 2>(x);
    } else {
        return x;
    }
}

// All-reduce over the 64 lanes (every lane gets the bit-identical result).
__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp<0xB1>(x));
    x = fmaxf(x, dpp<0x4E>(x));
    x = fmaxf(x, dpp<0x141>(x));
    x = fmaxf(x, dpp<0x140>(x));
    x = fmaxf(x, swizzle<0x401F>(x));
    x = fmaxf(x, lane_xor(x, 32));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp<0xB1>(x);
    x += dpp<0x4E>(x);
    x += dpp<0x141>(x);
    x += dpp<0x140>(x);
    x += swizzle<0x401F>(x);
    x += lane_xor(x, 32);
    return x;
}

// Partner value for step MASK of a butterfly inside a row group of G lanes.
// The first step (MASK == G/2) may pair lane s with G-1-s (a mirror, which
// DPP does cheaply); later steps must pair s with s ^ MASK exactly.
template <int G, int MASK>
__device__ __forceinline__ float group_partner(float x) {
    if constexpr (MASK == G / 2 && MASK == 4) return dpp<0x141>(x);   // row_half_mirror
    else if constexpr (MASK == G / 2 && MASK == 8) return dpp<0x140>(x);  // row_mirror
    else return xor_lane<MASK>(x);
}

// Reduce-scatter of the QK^T partial sums inside a row group of G lanes.
// On entry every lane holds, for the tile's NI row loads u and each beam i,
// its own 16-byte slice of the dot product d[u][i].  On exit d[j][i],
// j < max(1, NI/G), holds the complete dot product of row
// u = (sub / max(1, G/NI)) * max(1, NI/G) + j: the NI*KB sums are spread
// over the group instead of being repeated in every lane, so each score is
// turned into a probability once (G/NI times when G > NI).
template <int G, int KB, int NI, int MASK = G / 2, int NR = NI>
__device__ __forceinline__ void group_reduce_scatter(float (&d)[NI][KB], int sub) {
    if constexpr (MASK >= 1) {
        if constexpr (NR > 1) {
            constexpr int HALF = NR / 2;
            const bool up = (sub & MASK) != 0;
#pragma unroll
            for (int j = 0; j < HALF; ++j) {
#pragma unroll
                for (int i = 0; i < KB; ++i) {
                    const float send = up ? d[j][i] : d[j + HALF][i];
                    const float keep = up ? d[j + HALF][i] : d[j][i];
                    d[j][i] = keep + group_partner<G, MASK>(send);
                }
            }
            group_reduce_scatter<G, KB, NI, MASK / 2, HALF>(d, sub);
        } else {
#pragma unroll
            for (int i = 0; i < KB; ++i) d[0][i] += group_partner<G, MASK>(d[0][i]);
            group_reduce_scatter<G, KB, NI, MASK / 2, 1>(d, sub);
        }
    }
}

// Index of this wave in its workgroup, as a wave-uniform (scalar) value, so
// that branches on it are uniform and each side keeps its own registers.
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

__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

// Merge softmax state (mb, lb, ab) into (m, l, a); m in the base-2 domain.
__device__ __forceinline__ void merge_state(float &m, float &l, float &a, float mb, float lb, float ab) {
    const float mx = fmaxf(m, mb);
    const float ms = (mx == -INFINITY) ? 0.f : mx;
    const float fa = __builtin_amdgcn_exp2f(m - ms);
    const float fb = __builtin_amdgcn_exp2f(mb - ms);
    l = l * fa + lb * fb;
    a = a * fa + ab * fb;
    m = mx;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <bool BF16>
__device__ __forceinline__ void store_out(void *out, size_t idx, float v) {
    if constexpr (BF16)
        static_cast<uint16_t *>(out)[idx] = f32_to_bf16_rne(v);
    else
        static_cast<float *>(out)[idx] = v;
}

// Bound on re-reads of a partial-record word that does not yet carry the
// current call's tag (about 10 ms at most; not reached in practice).
constexpr int kMaxSpins = 1 << 14;

// State of one wave tile: keys [t0, min(t0 + kTile, j1)) of one K/V stream
// (t0 < j1), attended by the KB queries qr.  Kb/Vb point at row 0 of the
// stream (rows of kLpr 16-byte slices).  On return m[i], l[i] (base-2 max and
// sum of exp2) are wave-uniform and acc[i][e] holds, in every lane, the
// unnormalised output for dims sub*kEpl + e.  prow is this wave's LDS area.
// Rows of a generated-token tile read through an ancestry table: row j of
// the hypothesis is row j of the block of beam row[j] of its source (an entry
// outside [0, k) reads the hypothesis' own block, `self`).  The K/V pointers
// then address the source's beam-0 block, and `stride` is the distance in
// bytes between the blocks of two beams (H * T * row bytes).
struct Anc {
    const int32_t *row;
    int self, k, stride;
    // beams of this lane's rows of the first tile (t0 = 0), when `early`:
    // loaded before the tile, so that its K/V loads need not wait for them
    int first[kIt];
    bool early;
    __device__ __forceinline__ int beam(int j) const {
        const int a = row[j];
        return (a >= 0 && a < k) ? a : self;
    }
    // the beam of row j = t0 + u * rows-per-load + lane group, clamped to j1 - 1
    __device__ __forceinline__ int beam_at(int t0, int u, int j) const {
        return (early && t0 == 0) ? first[u] : beam(j);
    }
};

template <int D, bool BF16, int KB, bool IND = false>
__device__ __forceinline__ void tile_attend(const uint4 (&qr)[KB], const uint4 *__restrict__ Kb,
                                            const uint4 *__restrict__ Vb, int t0, int j1, int sub,
                                            int grp, float *prow, float scale_log2, float (&m)[KB],
                                            float (&l)[KB], float (&acc)[KB][Geo<D, BF16>::kEpl],
                                            const Anc &an = Anc{})
{
    using G = Geo<D, BF16>;
    constexpr int kEpl = G::kEpl, kLpr = G::kLpr, kRpi = G::kRpi;
    // Row loads: instruction u reads rows t0 + u*kRpi + grp.  Rows past j1
    // re-read row j1 - 1 (valid data, never padding) and are masked.
    uint4 kr[kIt], vr[kIt];
#pragma unroll
    for (int u = 0; u < kIt; ++u) {
        const int j = min(t0 + u * kRpi + grp, j1 - 1);
        size_t at = (size_t)j * kLpr + sub;
        if constexpr (IND) at += (size_t)an.beam_at(t0, u, j) * (an.stride / 16);
        kr[u] = load_nt(Kb + at);
        vr[u] = load_nt(Vb + at);
    }
    // QK^T: partial dots of this lane's slice, then a reduce-scatter in the
    // row group, after which the lane owns whole score rows.
    float d[kIt][KB];
#pragma unroll
    for (int u = 0; u < kIt; ++u) {
#pragma unroll
        for (int i = 0; i < KB; ++i) d[u][i] = dot16<BF16>(qr[i], kr[u], 0.f);
    }
    group_reduce_scatter<kLpr, KB, kIt>(d, sub);
    constexpr int kRows = G::kRows, kDup = G::kDup;
    const int u0 = (sub / kDup) * kRows;  // first score row of this lane
    float mt[KB];
#pragma unroll
    for (int i = 0; i < KB; ++i) {
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < kRows; ++j) {
            const bool ok = t0 + (u0 + j) * kRpi + grp < j1;
            d[j][i] = ok ? d[j][i] * scale_log2 : -INFINITY;
            mx = fmaxf(mx, d[j][i]);
        }
        mt[i] = wave_max(mx);  // tile maximum (finite: key t0 is valid)
    }
#pragma unroll
    for (int i = 0; i < KB; ++i) {
        float lsum = 0.f;
#pragma unroll
        for (int j = 0; j < kRows; ++j) {
            d[j][i] = __builtin_amdgcn_exp2f(d[j][i] - mt[i]);
            lsum += d[j][i];
        }
        l[i] = wave_sum(sub % kDup == 0 ? lsum : 0.f);
        m[i] = mt[i];
    }
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
        const int r = (u0 + j) * kRpi + grp;
#pragma unroll
        for (int i = 0; i < KB; ++i) prow[(r + (r >> 3)) * KB + i] = d[j][i];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // PV: the coalesced V rows with their weights read back from LDS
#pragma unroll
    for (int i = 0; i < KB; ++i) {
#pragma unroll
        for (int e = 0; e < kEpl; ++e) acc[i][e] = 0.f;
    }
#pragma unroll
    for (int u = 0; u < kIt; ++u) {
        const int r = u * kRpi + grp;
        float pw[KB];
#pragma unroll
        for (int i = 0; i < KB; ++i) pw[i] = prow[(r + (r >> 3)) * KB + i];
        float vf[kEpl];
        unpack16<BF16>(vr[u], vf);
#pragma unroll
        for (int i = 0; i < KB; ++i) {
#pragma unroll
            for (int e = 0; e < kEpl; ++e) acc[i][e] = fmaf(pw[i], vf[e], acc[i][e]);
        }
    }
    // the row groups hold partial sums of the same dims for different rows
#pragma unroll
    for (int i = 0; i < KB; ++i) {
#pragma unroll
        for (int e = 0; e < kEpl; ++e) acc[i][e] = groups_sum<kLpr>(acc[i][e]);
    }
    // keep the next tile's LDS writes behind this tile's reads
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Tag of the record words of a call, in their high 32 bits.  Outside graph
// capture the host passes an epoch in [1, 2^31).  A call captured into a
// graph passes 0 and takes, for each (b, h) row, that row's counter in the
// workspace with bit 31 set (so no host epoch equals it); the row's merger
// advances the counter once it has every record, so each replay of the
// graph tags its records anew.  c0 receives the counter value.
__device__ __forceinline__ unsigned long long call_tag(unsigned long long epoch, const unsigned long long *ctr,
                                                       unsigned long long &c0) {
    if (epoch != 0) return (epoch & 0xffffffffull) << 32;
    c0 = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return (0x80000000ull | ((c0 % 0x7fffffffull) + 1)) << 32;
}

// Store one record word (call tag << 32 | fp32 bits) with a device-scope atomic.
__device__ __forceinline__ void store_word(unsigned long long *p, unsigned long long tag, float v) {
    __hip_atomic_store(p, tag | __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// ---- tile policies -----------------------------------------------------------
// A policy attends one wave tile of keys and keeps one wave's softmax state
// per beam.  The kernels below only move these states through LDS and the
// workspace, so every decomposition of a call folds the same tile states in
// the same order.
//   ValuTile  fp32, and bf16 with D = 16: the VALU routine above.
//   MfmaTile  bf16 with D >= 32: both contractions on the matrix cores.

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));

template <int D, bool BF16, int KB>
struct ValuTile {
    using G = Geo<D, BF16>;
    static constexpr int kEpl = G::kEpl, kLpr = G::kLpr;
    static constexpr int kLdsBytes = G::kPStride * KB * 4;  // per wave
    struct Q { uint4 r[KB]; };
    static constexpr int kAStride = D;  // floats between the beams of a wave's state in LDS
    // m, l wave-uniform; acc[i][e] holds dims sub*kEpl + e in every lane
    struct St { float m[KB], l[KB], acc[KB][kEpl]; };

    // queries of hypotheses hyp0 .. hyp0 + KB - 1, head h
    static __device__ __forceinline__ void load_q(Q &q, const uint4 *__restrict__ qp, size_t hyp0, int h, int H,
                                                  int lane) {
        const int sub = lane % kLpr;
#pragma unroll
        for (int i = 0; i < KB; ++i) q.r[i] = qp[((hyp0 + i) * H + h) * kLpr + sub];
    }
    static __device__ __forceinline__ void init(St &s) {
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            s.m[i] = -INFINITY;
            s.l[i] = 0.f;
#pragma unroll
            for (int e = 0; e < kEpl; ++e) s.acc[i][e] = 0.f;
        }
    }
    template <bool IND = false>
    static __device__ __forceinline__ void attend(const Q &q, const uint4 *__restrict__ Kb,
                                                  const uint4 *__restrict__ Vb, int t0, int j1, int lane,
                                                  void *lds, float scale_log2, St &s, const Anc &an = Anc{}) {
        tile_attend<D, BF16, KB, IND>(q.r, Kb, Vb, t0, j1, lane % kLpr, lane / kLpr, static_cast<float *>(lds),
                                      scale_log2, s.m, s.l, s.acc, an);
    }
    // this wave's state into LDS: m_w[KB], l_w[KB], a_w[KB][D]
    static __device__ __forceinline__ void to_lds(const St &s, int lane, float *m_w, float *l_w, float *a_w) {
        if (lane < kLpr) {
#pragma unroll
            for (int i = 0; i < KB; ++i) {
#pragma unroll
                for (int e = 0; e < kEpl; ++e) a_w[i * kAStride + lane * kEpl + e] = s.acc[i][e];
            }
        }
        if (lane == 0) {
#pragma unroll
            for (int i = 0; i < KB; ++i) {
                m_w[i] = s.m[i];
                l_w[i] = s.l[i];
            }
        }
    }
};

// Value of x in lanes l & ~MASK and l | MASK (MASK = 16 or 32), in that
// order, in both lanes: combining the pair commutes nothing, so both lanes
// get bit-identical results.
template <int MASK>
__device__ __forceinline__ void lane_pair(float x, float &lo, float &hi) {
    const unsigned u = __float_as_uint(x);
    if constexpr (MASK == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        lo = __uint_as_float(r[0]);
        hi = __uint_as_float(r[1]);
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        lo = __uint_as_float(r[0]);
        hi = __uint_as_float(r[1]);
    }
}
// max / sum over the four lanes n, n + 16, n + 32, n + 48 of a column
__device__ __forceinline__ float col_max(float x) {
    float a, b;
    lane_pair<16>(x, a, b);
    x = fmaxf(a, b);
    lane_pair<32>(x, a, b);
    return fmaxf(a, b);
}
__device__ __forceinline__ float col_sum(float x) {
    float a, b;
    lane_pair<16>(x, a, b);
    x = a + b;
    lane_pair<32>(x, a, b);
    return a + b;
}

// bf16 tile on the matrix cores (v_mfma_f32_16x16x32_bf16; D = 32, 64, 128).
// The tile has T = 4096 / D keys (the row-load geometry of the VALU
// routine, so chunks are the same size).  K and V rows are loaded whole
// and coalesced, then pass through one swizzled LDS tile per wave (K first,
// then V in its place) to reach the operand layouts.  Lane l = 16 g + n:
//   QK^T  S^T[key][beam] = K[key][:] . q[beam][:]: the A operand is K
//         (lane: key 16 kb + n, 16 bytes at dim 32 s + 8 g), the B operand
//         the queries (column n = beam n < KB, the other columns zero).
//         Lane l gets the scores of beam n for keys 16 kb + 4 g + i.
//   softmax  per lane over its 4 NKB scores, then over the four lanes of
//         its column: every beam at once, no LDS.
//   PV    O^T[dim][beam] = V^T[dim][key] . P^T[key][beam].  P^T is the B
//         operand straight from the score registers (rounded to bf16; the
//         sum uses the rounded weights, so they add up to one).  V^T comes
//         from the tile's V rows staged in LDS and read back with
//         ds_read_b64_tr_b16, which transposes 16-bit elements within each
//         group of 16 lanes.  Lane l gets dims 16 mb + 4 g + i of beam n.
template <int D, int KB>
struct MfmaTile {
    static constexpr int T = 4096 / D;    // keys per tile
    static constexpr int NKB = T / 16;    // 16-key blocks
    static constexpr int NS = D / 32;     // 32-dim steps of QK^T
    static constexpr int NU = D / 16;     // 32-byte units per row = 16-dim output blocks
    static constexpr int kLpr = D / 8;    // 16-byte slices per row
    static constexpr int kLdsBytes = T * D * 2;  // one tile of rows (8 KB): K, then V
    static_assert(D == 32 || D == 64 || D == 128, "MFMA tile needs D in {32, 64, 128}");
    static_assert(KB <= 16, "beams are the 16 columns of the MFMA");
    static_assert(NKB % 2 == 0, "PV takes 32 keys per instruction");
    struct Q { bf16x8_t b[NS]; };
    // floats between the beams of a wave's state in LDS: the 16 lanes of one
    // store (one beam each) land on distinct banks (a stride of D puts them
    // all on the same four banks)
    static constexpr int kAStride = D + 4;
    // column state of beam n = lane & 15: m, l identical in the column's
    // four lanes; acc[mb][i] holds dim 16 mb + 4 (lane >> 4) + i
    struct St { float m, l; f32x4_t acc[NU]; };

    // 32-byte unit of row r holding unit c: a XOR swizzle that spreads the
    // 16 rows of one transposed read over all LDS banks
    static __device__ __forceinline__ int unit(int r, int c) {
        constexpr int sh = NU == 2 ? 2 : NU == 4 ? 1 : 0;
        return c ^ ((r >> sh) & (NU - 1));
    }
    static __device__ __forceinline__ void load_q(Q &q, const uint4 *__restrict__ qp, size_t hyp0, int h, int H,
                                                  int lane) {
        const int n = lane & 15, g = lane >> 4;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (n < KB) v = qp[((hyp0 + n) * H + h) * kLpr + 4 * s + g];
            q.b[s] = __builtin_bit_cast(bf16x8_t, v);
        }
    }
    static __device__ __forceinline__ void init(St &s) {
        s.m = -INFINITY;
        s.l = 0.f;
#pragma unroll
        for (int mb = 0; mb < NU; ++mb) s.acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    // row r of the tile (2 D bytes), 16-byte slice sl, in the swizzled LDS tile
    static __device__ __forceinline__ int lds_off(int r, int sl) {
        return r * (2 * D) + (unit(r, sl >> 1) << 5) + ((sl & 1) << 4);
    }
    static __device__ __forceinline__ void lds_fence() {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    template <bool IND = false>
    static __device__ __forceinline__ void attend(const Q &q, const uint4 *__restrict__ Kb,
                                                  const uint4 *__restrict__ Vb, int t0, int j1, int lane,
                                                  void *lds, float scale_log2, St &st, const Anc &an = Anc{}) {
        const int n = lane & 15, g = lane >> 4;
        // Row loads in the coalesced layout: kLpr lanes per row, so one
        // instruction reads whole rows (loads of 16 half rows each are
        // markedly slower).  Buffer loads whose range ends at row j1: rows
        // past it read as zero without a memory access and are masked, and
        // K and V share one offset register.  All K first, so its trip
        // through LDS can start while V is in flight.
        constexpr int kRpi = kWave / kLpr;
        const int sub = lane % kLpr, grp = lane / kLpr;
        uint4 kr[kIt], vr[kIt];
        if constexpr (!IND) {
            const auto kres = row_rsrc(Kb, j1 * 2 * D), vres = row_rsrc(Vb, j1 * 2 * D);
            const int off = ((t0 + grp) * kLpr + sub) * 16;
#pragma unroll
            for (int u = 0; u < kIt; ++u) kr[u] = load_rows(kres, off, u * kRpi * 2 * D);
#pragma unroll
            for (int u = 0; u < kIt; ++u) vr[u] = load_rows(vres, off, u * kRpi * 2 * D);
        } else {
            // each row from its beam's block; rows at or past j1 get an
            // offset past the range and read zero without a memory access
            const auto kres = row_rsrc(Kb, an.k * an.stride), vres = row_rsrc(Vb, an.k * an.stride);
            int off[kIt];
#pragma unroll
            for (int u = 0; u < kIt; ++u) {
                const int j = t0 + grp + u * kRpi;
                const int a = an.beam_at(t0, u, min(j, j1 - 1));
                off[u] = j < j1 ? a * an.stride + (j * kLpr + sub) * 16 : 0x7ffffff0;
            }
#pragma unroll
            for (int u = 0; u < kIt; ++u) kr[u] = load_rows(kres, off[u], 0);
#pragma unroll
            for (int u = 0; u < kIt; ++u) vr[u] = load_rows(vres, off[u], 0);
        }
        // K through LDS into the MFMA A layout: lane l takes row 16 kb + n,
        // dims 32 s + 8 g .. + 8
        char *vt = static_cast<char *>(lds);
#pragma unroll
        for (int u = 0; u < kIt; ++u) *reinterpret_cast<uint4 *>(vt + lds_off(u * kRpi + grp, sub)) = kr[u];
        lds_fence();
        uint4 ka[NKB][NS];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
            for (int s = 0; s < NS; ++s) ka[kb][s] = *reinterpret_cast<const uint4 *>(vt + lds_off(16 * kb + n, 4 * s + g));
        }
        lds_fence();
        // the V rows take the K rows' place (this wave's reads of K are done:
        // LDS instructions of one wave complete in order)
#pragma unroll
        for (int u = 0; u < kIt; ++u) *reinterpret_cast<uint4 *>(vt + lds_off(u * kRpi + grp, sub)) = vr[u];
        f32x4_t sc[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            sc[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < NS; ++s)
                sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[kb][s]), q.b[s],
                                                                 sc[kb], 0, 0, 0);
        }
        // scores in the base-2 domain; keys past j1 get weight zero
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool ok = t0 + 16 * kb + 4 * g + i < j1;
                sc[kb][i] = ok ? sc[kb][i] * scale_log2 : -INFINITY;
                mx = fmaxf(mx, sc[kb][i]);
            }
        }
        mx = col_max(mx);  // finite: key t0 is valid
        bf16x8_t pb[NKB / 2];
        float ls = 0.f;
#pragma unroll
        for (int pp = 0; pp < NKB / 2; ++pp) {
            f32x8_t e;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                e[i] = __builtin_amdgcn_exp2f(sc[2 * pp][i] - mx);
                e[4 + i] = __builtin_amdgcn_exp2f(sc[2 * pp + 1][i] - mx);
            }
            pb[pp] = __builtin_convertvector(e, bf16x8_t);
#pragma unroll
            for (int i = 0; i < 8; ++i) ls += (float)pb[pp][i];
        }
        ls = col_sum(ls);
        lds_fence();
        // PV: MFMA pp contracts over keys [32 pp, 32 pp + 32) in the order
        // the score registers hold them: k = 8 g + j stands for key
        // 16 (2 pp + j / 4) + 4 g + j % 4.
        f32x4_t o[NU];
#pragma unroll
        for (int mb = 0; mb < NU; ++mb) o[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int pp = 0; pp < NKB / 2; ++pp) {
#pragma unroll
            for (int mb = 0; mb < NU; ++mb) {
                i16x4_t t[2];
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int row = 32 * pp + 16 * r + 4 * g + (n >> 2);
                    const int off = row * (2 * D) + (unit(row, mb) << 5) + ((n & 3) << 3);
                    t[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) i16x4_t *)(vt + off));
                }
                const auto a = __builtin_shufflevector(t[0], t[1], 0, 1, 2, 3, 4, 5, 6, 7);
                o[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), pb[pp], o[mb],
                                                                0, 0, 0);
            }
        }
        // keep the next tile's LDS writes behind this tile's reads
        lds_fence();
        st.m = mx;
        st.l = ls;
#pragma unroll
        for (int mb = 0; mb < NU; ++mb) st.acc[mb] = o[mb];
    }
    static __device__ __forceinline__ void to_lds(const St &s, int lane, float *m_w, float *l_w, float *a_w) {
        const int n = lane & 15, g = lane >> 4;
        if (n < KB) {
#pragma unroll
            for (int mb = 0; mb < NU; ++mb)
                *reinterpret_cast<f32x4_t *>(a_w + n * kAStride + 16 * mb + 4 * g) = s.acc[mb];
            if (g == 0) {
                m_w[n] = s.m;
                l_w[n] = s.l;
            }
        }
    }
};

template <int D, bool BF16, int KB>
using Tile = typename std::conditional<(BF16 && D >= 32), MfmaTile<D, KB>, ValuTile<D, BF16, KB>>::type;

// LDS area of one wave: large enough for a tile of KB beams or of one beam,
// for the wave's acc (KB rows of kAStride floats) once its tile is done, and for one generated-
// token tile state (m, l, acc[D] at float 4); a 16-byte multiple.
template <int D, bool BF16, int KB>
struct WaveLds {
    static constexpr int a = Tile<D, BF16, KB>::kLdsBytes, b = Tile<D, BF16, 1>::kLdsBytes;
    static constexpr int s = Tile<D, BF16, KB>::kAStride;
    static constexpr int c = KB * s * 4 > (D + 4) * 4 ? KB * s * 4 : (D + 4) * 4;
    static constexpr int kBytes = ((a > b ? (a > c ? a : c) : (b > c ? b : c)) + 15) / 16 * 16;
};


// Merger for (b, h) = bh: merges the chunk records of a source with more
// than one chunk, in chunk order, and writes the normalised output.
//
// Each record word is (call tag << 32 | fp32 bits), written and read with
// device-scope atomics: every word is coherent across XCDs by itself, and
// the tag tells whether it was written by this call, so no fence or counter
// is needed.  The chunk workgroups have lower ids and were dispatched
// earlier, and they wait on nothing, so their records arrive; a word that
// does not carry this call's tag yet is re-read a bounded number of times,
// and the output becomes NaN if it never does (a loud failure instead of a
// silent wrong merge or an endless wait).
//
// The records are the row's tile states, one per tile of keys in key order
// (record slot j holds tile j), folded one by one from the empty state.
// With a generated-token segment (SPLIT), record slot NT of (b, h) holds the
// per-beam state of that segment; it is merged after the prefix tiles, and
// the merger also writes the rows whose prefix has at most one chunk.
template <int D, bool BF16, int KB, bool SPLIT>
__device__ __forceinline__ void merge_chunks(const unsigned long long *__restrict__ part,
                                             const int32_t *__restrict__ src_len, void *__restrict__ out,
                                             int bh, int n_bh, int H, int S, int NT, int t,
                                             unsigned long long epoch, unsigned long long *__restrict__ ctr)
{
    using G = Geo<D, BF16>;
    if (bh >= n_bh) return;
    const int b = bh / H;
    const int h = bh - b * H;
    const int L = min(max(src_len[b], 0), S);
    if (!SPLIT && (L + G::kChunk - 1) / G::kChunk <= 1) return;  // written by the chunk workgroup itself
    const int nc = (L + G::kTile - 1) / G::kTile;             // tile records of the prefix, in key order
    const int nrec = nc + (SPLIT && t > 0 ? 1 : 0);          // records to merge, in order
    constexpr int kRec = KB * (D + 2);
    unsigned long long c0 = 0;
    const unsigned long long tag = call_tag(epoch, ctr + bh, c0);
    const unsigned long long *recs = part + (size_t)bh * (NT + (SPLIT ? 1 : 0)) * kRec;
    bool stale_any = false;
    const size_t obase = ((size_t)b * KB * H + h) * D;
    constexpr int kBatch = 4;  // records whose words are loaded together
    for (int x = threadIdx.x; x < KB * D; x += kBlock) {
        const int i = x / D, d = x - i * D;
        const int at[3] = {KB * D + i, KB * D + KB + i, x};  // m, l, acc
        float mm = -INFINITY, ll = 0.f, aa = 0.f;
        bool stale = false;
        for (int c0 = 0; c0 < nrec; c0 += kBatch) {
            unsigned long long wv[kBatch][3];
#pragma unroll
            for (int q2 = 0; q2 < kBatch; ++q2) {
                // the generated-token record sits in slot NT
                const int slot = (SPLIT && c0 + q2 == nc) ? NT : c0 + q2;
#pragma unroll
                for (int f = 0; f < 3; ++f) {
                    wv[q2][f] = tag;
                    if (c0 + q2 < nrec)
                        wv[q2][f] = __hip_atomic_load(recs + (size_t)slot * kRec + at[f],
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
#pragma unroll
            for (int q2 = 0; q2 < kBatch; ++q2) {
                if (c0 + q2 >= nrec) break;
                const int slot = (SPLIT && c0 + q2 == nc) ? NT : c0 + q2;
#pragma unroll
                for (int f = 0; f < 3; ++f) {
                    const unsigned long long *a = recs + (size_t)slot * kRec + at[f];
                    for (int spin = 0; (wv[q2][f] & 0xffffffff00000000ull) != tag && spin < kMaxSpins; ++spin) {
                        __builtin_amdgcn_s_sleep(2);
                        wv[q2][f] = __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                    stale |= (wv[q2][f] & 0xffffffff00000000ull) != tag;
                }
                merge_state(mm, ll, aa, __uint_as_float((uint32_t)wv[q2][0]),
                            __uint_as_float((uint32_t)wv[q2][1]), __uint_as_float((uint32_t)wv[q2][2]));
            }
        }
        const float o = nrec == 0 ? 0.f : aa / ll;  // no key at all: zero row
        store_out<BF16>(out, obase + (size_t)i * H * D + d, stale ? NAN : o);
        stale_any |= stale;
    }
    // a captured call: every record of the row is in (or the wait ran out),
    // so every workgroup of the row has read the counter; the next call takes
    // the next value (skipping one after a wait that ran out, so that a late
    // record of this call can never pass for the next call's)
    const int any = __syncthreads_or(stale_any);
    if (epoch == 0 && threadIdx.x == 0)
        __hip_atomic_store(ctr + bh, c0 + (any ? 2 : 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Softmax state of one hypothesis over its generated rows, in the compact
// layout: m, l in every lane, lane l holding acc for dims l, l + 64, ...
template <int D>
struct GenState {
    static constexpr int kE = (D + kWave - 1) / kWave;
    float m, l, a[kE];
};

// Softmax state of hypothesis `hyp` over its own generated rows [0, t) of
// Kt/Vt for head h (t > 0): the tiles in order, each folded into the running
// state.  Each tile's state passes through the wave's LDS area (m, l, then
// acc[D] at float 4), so the running state takes a few registers per lane
// rather than a whole tile state.
template <int D, bool BF16, bool IND>
__device__ __forceinline__ void generated_fold(const uint4 *__restrict__ q, const uint4 *__restrict__ Kb,
                                               const uint4 *__restrict__ Vb, size_t hyp, int h, int H, int t,
                                               int lane, void *lds, float scale_log2, GenState<D> &gs,
                                               const Anc &an)
{
    using TL = Tile<D, BF16, 1>;
    constexpr int kTile = Geo<D, BF16>::kTile, kE = GenState<D>::kE;
    typename TL::Q qv;
    TL::load_q(qv, q, hyp, h, H, lane);
    float *slot = static_cast<float *>(lds);
    gs.m = -INFINITY;
    gs.l = 0.f;
#pragma unroll
    for (int e = 0; e < kE; ++e) gs.a[e] = 0.f;
    for (int t0 = 0; t0 < t; t0 += kTile) {
        typename TL::St ts;
        TL::template attend<IND>(qv, Kb, Vb, t0, t, lane, lds, scale_log2, ts, an);
        TL::to_lds(ts, lane, slot, slot + 1, slot + 4);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // fold the tile into the running state (the order of merge_state)
        const float tm = slot[0], tl = slot[1];
        const float mx = fmaxf(gs.m, tm);
        const float ms = (mx == -INFINITY) ? 0.f : mx;
        const float fa = __builtin_amdgcn_exp2f(gs.m - ms);
        const float fb = __builtin_amdgcn_exp2f(tm - ms);
        gs.l = gs.l * fa + tl * fb;
#pragma unroll
        for (int e = 0; e < kE; ++e) {
            const int d = lane + e * kWave;
            if (d < D) gs.a[e] = gs.a[e] * fa + slot[4 + d] * fb;
        }
        gs.m = mx;
        // the next tile's LDS writes stay behind these reads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// Beam `self` of a source, hypothesis hyp = source * k + self: its state over
// its generated rows [0, t) of head h.  Without a table they are rows of its
// own block of Kt/Vt; with an ancestry row (anc_row[j] = the beam whose block
// holds its row j) each row comes from that beam's block.
template <int D, bool BF16, bool ANC>
__device__ __forceinline__ void generated_state(const uint4 *__restrict__ q, const uint4 *__restrict__ Kt,
                                                const uint4 *__restrict__ Vt, size_t hyp, int h, int H, int T,
                                                int t, int lane, void *lds, float scale_log2, GenState<D> &gs,
                                                const int32_t *anc_row, int self, int k,
                                                const int (&first)[kIt] = {}, bool early = false)
{
    constexpr int kLpr = Geo<D, BF16>::kLpr;
    if constexpr (ANC) {
        const size_t base = ((hyp - self) * H + h) * (size_t)T * kLpr;   // the source's beam-0 block
        Anc an{anc_row, self, k, H * T * kLpr * 16};
        an.early = early;
#pragma unroll
        for (int u = 0; u < kIt; ++u) an.first[u] = first[u];
        generated_fold<D, BF16, true>(q, Kt + base, Vt + base, hyp, h, H, t, lane, lds, scale_log2, gs, an);
    } else {
        const size_t base = (hyp * H + h) * (size_t)T * kLpr;
        generated_fold<D, BF16, false>(q, Kt + base, Vt + base, hyp, h, H, t, lane, lds, scale_log2, gs, Anc{});
    }
}

// Generated-token segment of (b, h) = bh (SPLIT only): wave w attends beam
// i = w, w + 4, ... over that hypothesis' own rows [0, t) of Kt/Vt and stores
// the beam's state in record slot NC of (b, h).
template <int D, bool BF16, int KB, bool ANC>
__device__ __forceinline__ void attend_generated(const uint4 *__restrict__ q, const uint4 *__restrict__ Kt,
                                                 const uint4 *__restrict__ Vt, unsigned long long *__restrict__ part,
                                                 int bh, int n_bh, int H, int NT, int T, int t,
                                                 float scale_log2, unsigned long long epoch,
                                                 const unsigned long long *__restrict__ ctr, void *lds,
                                                 const int32_t *__restrict__ anc, int ld_anc)
{
    if (bh >= n_bh || t <= 0) return;
    const int b = bh / H;
    const int h = bh - b * H;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_id();
    constexpr int kRec = KB * (D + 2);
    unsigned long long c0;
    const unsigned long long tag = call_tag(epoch, ctr + bh, c0);
    unsigned long long *rec = part + ((size_t)bh * (NT + 1) + NT) * kRec;
    for (int i = w; i < KB; i += kWaves) {
        GenState<D> gs;
        const size_t hyp = (size_t)b * KB + i;
        generated_state<D, BF16, ANC>(q, Kt, Vt, hyp, h, H, T, t, lane, lds, scale_log2, gs,
                                      ANC ? anc + hyp * ld_anc : nullptr, i, KB);
#pragma unroll
        for (int e = 0; e < GenState<D>::kE; ++e) {
            const int d = lane + e * kWave;
            if (d < D) store_word(rec + i * D + d, tag, gs.a[e]);
        }
        if (lane == 0) {
            store_word(rec + KB * D + i, tag, gs.m);
            store_word(rec + KB * D + KB + i, tag, gs.l);
        }
    }
}

template <int D, bool BF16, int KB, bool SPLIT, bool ANC = false>
__global__ __launch_bounds__(kBlock) void cross_attn_kernel(
    const uint4 *__restrict__ q, const uint4 *__restrict__ K, const uint4 *__restrict__ V,
    const int32_t *__restrict__ src_len, void *__restrict__ out,
    unsigned long long *__restrict__ part,
    int n_bh, int H, int S, int NC, float scale_log2, unsigned long long epoch,
    unsigned long long *__restrict__ ctr,
    const uint4 *__restrict__ Kt, const uint4 *__restrict__ Vt, int T, int t, const int32_t *__restrict__ anc,
    int ld_anc, NgramJob ngj)
{
    using G = Geo<D, BF16>;
    using TL = Tile<D, BF16, KB>;
    constexpr int kLpr = G::kLpr;
    constexpr int kTile = G::kTile, kChunk = G::kChunk;

    // A fused decode step's n-gram rows take the first workgroups (a
    // multiple of 8, so the XCD residues of the ids below are kept).
    if ((int)blockIdx.x < ngj.blocks) {
        ngram_job_block(ngj, blockIdx.x, kWaves);
        return;
    }

    __shared__ float m_lds[kWaves][KB], l_lds[kWaves][KB];
    // each wave's tile area, which then holds its acc[KB][D] for the merge
    __shared__ __attribute__((aligned(16))) char t_lds[kWaves][WaveLds<D, BF16, KB>::kBytes];
    auto a_lds = [&](int ww) { return reinterpret_cast<float *>(&t_lds[ww][0]); };

    // Workgroup g runs on XCD g % 8 (round-robin dispatch).  All chunks of
    // one (b, h), its generated-token workgroup and its merger get ids with
    // the same residue, so they share an L2.  Order of the id ranges: the
    // generated-token workgroups (SPLIT only; each walks its tiles in
    // sequence, so they start first), the chunk workgroups, the mergers.
    const int n_bh8 = ((n_bh + kXcds - 1) / kXcds) * kXcds;
    int g = blockIdx.x - ngj.blocks;
    if constexpr (SPLIT) {
        if (g < n_bh8) {
            attend_generated<D, BF16, KB, ANC>(q, Kt, Vt, part, g, n_bh, H, NC * kWaves, T, t, scale_log2, epoch,
                                               ctr, &t_lds[wave_id()][0], anc, ld_anc);
            return;
        }
        g -= n_bh8;
    }
    const int n_chunk_blocks = n_bh8 * NC;
    if (g >= n_chunk_blocks) {
        merge_chunks<D, BF16, KB, SPLIT>(part, src_len, out, g - n_chunk_blocks, n_bh, H, S, NC * kWaves, t, epoch,
                                         ctr);
        return;
    }
    const int xcd = g % kXcds;
    const int slot = g / kXcds;
    const int bh = (slot / NC) * kXcds + xcd;
    const int c = slot - (slot / NC) * NC;
    if (bh >= n_bh) return;
    const int b = bh / H;
    const int h = bh - b * H;
    const int L = min(max(src_len[b], 0), S);
    const int j0 = c * kChunk;
    const int nc = (L + kChunk - 1) / kChunk;
    const int tid = threadIdx.x;
    const size_t obase = ((size_t)b * KB * H + h) * D;  // out[b, 0, h, 0]
    if (!SPLIT && L == 0) {  // no valid key: the output row is zero
        if (c == 0)
            for (int x = tid; x < KB * D; x += kBlock)
                store_out<BF16>(out, obase + (size_t)(x / D) * H * D + x % D, 0.f);
        return;
    }
    if (c >= nc) return;  // chunk lies in the padding: never read
    const int j1 = min(j0 + kChunk, L);
    // the call's tag (for a captured call a load, issued before the row's)
    unsigned long long c0;
    const unsigned long long tag = call_tag(epoch, ctr + bh, c0);

    const int lane = tid & (kWave - 1);
    const int w = wave_id();

    typename TL::Q qv;
    TL::load_q(qv, q, (size_t)b * KB, h, H, lane);
    const uint4 *Kbh = K + (size_t)bh * S * kLpr;
    const uint4 *Vbh = V + (size_t)bh * S * kLpr;

    typename TL::St st;
    TL::init(st);
    const int t0 = j0 + w * kTile;
    if (t0 < j1) TL::attend(qv, Kbh, Vbh, t0, j1, lane, &t_lds[w][0], scale_log2, st);
    TL::to_lds(st, lane, &m_lds[w][0], &l_lds[w][0], a_lds(w));
    __syncthreads();

    if (!SPLIT && nc == 1) {
        // the whole row: its tile states folded in key order from the empty state
        for (int x = tid; x < KB * D; x += kBlock) {
            const int i = x / D, d = x - i * D;
            float mm = -INFINITY, ll = 0.f, aa = 0.f;
#pragma unroll
            for (int ww = 0; ww < kWaves; ++ww)
                merge_state(mm, ll, aa, m_lds[ww][i], l_lds[ww][i], a_lds(ww)[i * TL::kAStride + d]);
            store_out<BF16>(out, obase + (size_t)i * H * D + d, aa / ll);
        }
        return;
    }

    // One record per tile of the chunk (slot = tile index in the row):
    // acc[KB][D], then m[KB], then l[KB].
    const int NT = NC * kWaves;
    const int ntile = min(kWaves, (j1 - j0 + kTile - 1) / kTile);   // tiles of this chunk that hold keys
    for (int ww = 0; ww < ntile; ++ww) {
        unsigned long long *rec = part + ((size_t)bh * (NT + (SPLIT ? 1 : 0)) + c * kWaves + ww) * (KB * (D + 2));
        for (int x = tid; x < KB * D; x += kBlock) {
            const int i = x / D, d = x - i * D;
            store_word(rec + x, tag, a_lds(ww)[i * TL::kAStride + d]);
            if (d == 0) {
                store_word(rec + KB * D + i, tag, m_lds[ww][i]);
                store_word(rec + KB * D + KB + i, tag, l_lds[ww][i]);
            }
        }
    }
}

// One workgroup per (b, h) that walks all of its chunks itself: no partial
// records, no merger, no cross-workgroup wait.  The row's jobs -- its chunks
// and, for the split cache, the generated tokens -- are processed P at a
// time by P groups of kWaves waves (workgroup of P*kBlock threads).  The
// generated-token job goes first, so that its tiles are read alongside the
// first chunks, but it is folded last.  The arithmetic and its order are
// those of cross_attn_kernel -- each chunk's four wave states merged in wave
// order, the chunk states folded in chunk order from the empty state, the
// generated-token state last -- so both kernels give the same bits.  It pays
// when there are enough (b, h) rows to fill the chip without splitting them.
template <int D, bool BF16, int KB, bool SPLIT, int P, bool ANC = false>
__global__ __launch_bounds__(kBlock * P) void attn_whole_kernel(
    const uint4 *__restrict__ q, const uint4 *__restrict__ K, const uint4 *__restrict__ V,
    const int32_t *__restrict__ src_len, void *__restrict__ out, int n_bh, int H, int S,
    float scale_log2, const uint4 *__restrict__ Kt, const uint4 *__restrict__ Vt, int T, int t,
    const int32_t *__restrict__ anc, int ld_anc, NgramJob ngj)
{
    using G = Geo<D, BF16>;
    using TL = Tile<D, BF16, KB>;
    constexpr int kLpr = G::kLpr;
    constexpr int kTile = G::kTile, kChunk = G::kChunk;
    constexpr int kW = kWaves * P;                        // waves per workgroup
    constexpr int kThreads = kBlock * P;
    constexpr int kPer = (KB * D + kThreads - 1) / kThreads;  // outputs per thread
    constexpr int kGB = SPLIT ? KB : 1, kGD = SPLIT ? D : 1;

    __shared__ float m_lds[kW][KB], l_lds[kW][KB];
    // each wave's tile area, which then holds its acc[KB][D] for the merge
    __shared__ __attribute__((aligned(16))) char t_lds[kW][WaveLds<D, BF16, KB>::kBytes];
    // generated-token states, kept until they are folded in at the end
    __shared__ __attribute__((aligned(16))) float g_lds[kGB][kGD];
    __shared__ float gm_lds[kGB], gl_lds[kGB];

    // A fused decode step's n-gram rows take the first workgroups.
    if ((int)blockIdx.x < ngj.blocks) {
        ngram_job_block(ngj, blockIdx.x, kW);
        return;
    }
    const int bh = blockIdx.x - ngj.blocks;
    if (bh >= n_bh) return;
    // trace words: 0 start, 1 end, 2 hardware ids, 3 row, 4 jobs, 5 first round folded
    unsigned long long *trs = trace_slot();
    trace::stamp(trs, 0);
    const int b = bh / H;
    const int h = bh - b * H;
    const int L = min(max(src_len[b], 0), S);
    const int nc = (L + kChunk - 1) / kChunk;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = wave_id();
    const size_t obase = ((size_t)b * KB * H + h) * D;  // out[b, 0, h, 0]
    // Through an ancestry table, the waves that take the generated-token job
    // (first group, round 0) load the beams of their first tile's rows now,
    // alongside src_len, instead of in front of the tile's K/V loads.
    int first[kIt] = {};
    bool early = false;
    if constexpr (SPLIT && ANC) {
        const int wg = wave_id();
        if (t > 0 && wg < kWaves && wg < KB) {
            const int32_t *row = anc + ((size_t)b * KB + wg) * ld_anc;
            const int grp = (int)(threadIdx.x & (kWave - 1)) / kLpr;
#pragma unroll
            for (int u = 0; u < kIt; ++u) {
                const int a = row[min(grp + u * G::kRpi, t - 1)];
                first[u] = (a >= 0 && a < KB) ? a : wg;
            }
            early = true;
        }
    }

    typename TL::Q qv;
    TL::load_q(qv, q, (size_t)b * KB, h, H, lane);
    const uint4 *Kbh = K + (size_t)bh * S * kLpr;
    const uint4 *Vbh = V + (size_t)bh * S * kLpr;

    // running state of output x = tid + p * kThreads (beam x / D, dim x % D)
    float Rm[kPer], Rl[kPer], Ra[kPer];
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
        Rm[p] = -INFINITY;
        Rl[p] = 0.f;
        Ra[p] = 0.f;
    }

    // jobs: [generated tokens (SPLIT, t > 0)] chunk 0, chunk 1, ...
    const int ng = (SPLIT && t > 0) ? 1 : 0;
    const int njobs = nc + ng;
    const int cg = w / kWaves;   // group of this wave: job j0 + cg of each step
    const int wt = w % kWaves;   // its wave in the group

    // The first group takes the generated-token job (job 0 of round 0) here,
    // before the job loop: its state stays out of the loop's registers (and
    // beams loaded early from an ancestry table die before it).
    if constexpr (SPLIT) {
        if (ng && cg == 0) {
            for (int i = wt; i < KB; i += kWaves) {
                GenState<D> gs;
                const size_t hyp = (size_t)b * KB + i;
                generated_state<D, BF16, ANC>(q, Kt, Vt, hyp, h, H, T, t, lane, &t_lds[w][0], scale_log2, gs,
                                              ANC ? anc + hyp * ld_anc : nullptr, i, KB, first, early && i == wt);
#pragma unroll
                for (int e = 0; e < GenState<D>::kE; ++e) {
                    const int d = lane + e * kWave;
                    if (d < D) g_lds[i][d] = gs.a[e];
                }
                if (lane == 0) {
                    gm_lds[i] = gs.m;
                    gl_lds[i] = gs.l;
                }
            }
        }
    }
    for (int j0 = 0; j0 < njobs; j0 += P) {
        const int c = j0 + cg - ng;  // chunk of this group's job; -1: generated tokens
        if (j0 + cg < njobs && c < 0) {
            // the generated-token job, already taken before this loop
        } else if (j0 + cg < njobs) {
            typename TL::St st;
            TL::init(st);
            const int j1 = min((c + 1) * kChunk, L);
            const int t0 = c * kChunk + wt * kTile;
            if (t0 < j1) TL::attend(qv, Kbh, Vbh, t0, j1, lane, &t_lds[w][0], scale_log2, st);
            TL::to_lds(st, lane, &m_lds[w][0], &l_lds[w][0], reinterpret_cast<float *>(&t_lds[w][0]));
        }
        __syncthreads();
#pragma unroll
        for (int p = 0; p < kPer; ++p) {
            const int x = tid + p * kThreads;
            if (x < KB * D) {
                const int i = x / D, d = x - i * D;
                for (int g = 0; g < P && j0 + g < njobs; ++g) {
                    if (j0 + g < ng) continue;  // the generated-token job is folded last
                    // the chunk's tile states, in key order (a tile past the
                    // row's end holds the empty state, which folds to nothing)
#pragma unroll
                    for (int ww = 0; ww < kWaves; ++ww) {
                        const int w0 = g * kWaves + ww;
                        const float *aw = reinterpret_cast<const float *>(&t_lds[w0][0]);
                        merge_state(Rm[p], Rl[p], Ra[p], m_lds[w0][i], l_lds[w0][i], aw[i * TL::kAStride + d]);
                    }
                }
            }
        }
        __syncthreads();
        if (j0 == 0) trace::stamp(trs, 5);
    }
    if (ng) {
#pragma unroll
        for (int p = 0; p < kPer; ++p) {
            const int x = tid + p * kThreads;
            if (x < KB * D) {
                const int i = x / D, d = x - i * D;
                merge_state(Rm[p], Rl[p], Ra[p], gm_lds[i], gl_lds[i], g_lds[i][d]);
            }
        }
    }
    const bool any = njobs > 0;
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
        const int x = tid + p * kThreads;
        if (x < KB * D) {
            const int i = x / D, d = x - i * D;
            store_out<BF16>(out, obase + (size_t)i * H * D + d, any ? Ra[p] / Rl[p] : 0.f);  // no key: zero row
        }
    }
    trace::stamp(trs, 1);
    trace::put(trs, 2, trace::where());
    trace::put(trs, 3, (unsigned long long)bh);
    trace::put(trs, 4, (unsigned long long)njobs);
}

// Launch arguments shared by both entry points.  For the encoder-decoder
// form Kt/Vt are null and T = t = 0.
struct AttnArgs {
    const void *q, *K, *V;
    const int32_t *src_len;
    void *out;
    int B, k, H, S, D;
    const void *Kt, *Vt;
    int T, t;
    const int32_t *anc;   // ancestry table of the generated rows, or null
    int ld_anc;
    float *ws;
    unsigned long long epoch;
    hipStream_t stream;
    NgramJob ng;          // n-gram rows of a fused decode step (ng.rows == 0: none)
    AttnPath path;        // decomposition chosen for the call
};

template <int D, bool BF16, int KB, bool SPLIT, bool ANC = false>
hipError_t launch_split(const AttnArgs &a, int NC)
{
    const int n_bh = a.B * a.H;
    const long long n_bh8 = ((long long)n_bh + kXcds - 1) / kXcds * kXcds;
    const double scale_log2 = 1.4426950408889634074 / sqrt((double)D);
    unsigned long long *part = reinterpret_cast<unsigned long long *>(a.ws);
    // the rows' counters for captured calls follow the records
    unsigned long long *ctr = part + (size_t)n_bh * (NC * kWaves + (SPLIT ? 1 : 0)) * (KB * (D + 2));
    // [generated-token workgroups] [chunk workgroups] [mergers]
    const long long mergers = (SPLIT || NC > 1) ? n_bh : 0;
    // n-gram workgroups first, rounded to a multiple of 8 so that the XCD
    // residues of the ids after them are kept
    NgramJob ng = a.ng;
    ng.blocks = ng.rows > 0 ? (ng.rows + kWaves - 1) / kWaves : 0;
    ng.blocks = (ng.blocks + kXcds - 1) / kXcds * kXcds;
    const long long nblk = ng.blocks + (SPLIT ? n_bh8 : 0) + n_bh8 * NC + mergers;
    hipLaunchKernelGGL((cross_attn_kernel<D, BF16, KB, SPLIT, ANC>), dim3((unsigned)nblk), dim3(kBlock), 0,
                       a.stream, static_cast<const uint4 *>(a.q), static_cast<const uint4 *>(a.K),
                       static_cast<const uint4 *>(a.V), a.src_len, a.out, part, n_bh, a.H, a.S,
                       NC, (float)scale_log2, a.epoch, ctr, static_cast<const uint4 *>(a.Kt),
                       static_cast<const uint4 *>(a.Vt), a.T, a.t, a.anc, a.ld_anc, ng);
    return hipGetLastError();
}

template <int D, bool BF16, int KB, bool SPLIT, int P, bool ANC = false>
hipError_t launch_whole(const AttnArgs &a)
{
    const int n_bh = a.B * a.H;
    const double scale_log2 = 1.4426950408889634074 / sqrt((double)D);
    NgramJob ng = a.ng;
    ng.blocks = ng.rows > 0 ? (ng.rows + kWaves * P - 1) / (kWaves * P) : 0;
    hipLaunchKernelGGL((attn_whole_kernel<D, BF16, KB, SPLIT, P, ANC>), dim3((unsigned)(ng.blocks + n_bh)),
                       dim3(kBlock * P), 0,
                       a.stream, static_cast<const uint4 *>(a.q), static_cast<const uint4 *>(a.K),
                       static_cast<const uint4 *>(a.V), a.src_len, a.out, n_bh, a.H, a.S, (float)scale_log2,
                       static_cast<const uint4 *>(a.Kt), static_cast<const uint4 *>(a.Vt), a.T, a.t, a.anc,
                       a.ld_anc, ng);
    return hipGetLastError();
}

template <int D, bool BF16, int KB, bool SPLIT>
hipError_t launch_typed(const AttnArgs &a)
{
    using G = Geo<D, BF16>;
    // at least one chunk column, so that a source with no valid key (or
    // S == 0) still has a workgroup to write its zero output
    const int NC = max(1, (a.S + G::kChunk - 1) / G::kChunk);
    const AttnPath path = a.path;
    if constexpr (SPLIT) {
        if (a.anc) {
            // generated rows through the ancestry table: their own kernels,
            // so that the table-free ones keep their registers
            switch (path) {
            case AttnPath::kWhole1: return launch_whole<D, BF16, KB, true, 1, true>(a);
            case AttnPath::kWhole2: return launch_whole<D, BF16, KB, true, 2, true>(a);
            case AttnPath::kWhole4: return launch_whole<D, BF16, KB, true, 4, true>(a);
            default: return launch_split<D, BF16, KB, true, true>(a, NC);
            }
        }
    }
    switch (path) {
    case AttnPath::kWhole1: return launch_whole<D, BF16, KB, SPLIT, 1>(a);
    case AttnPath::kWhole2: return launch_whole<D, BF16, KB, SPLIT, 2>(a);
    case AttnPath::kWhole4: return launch_whole<D, BF16, KB, SPLIT, 4>(a);
    default: return launch_split<D, BF16, KB, SPLIT>(a, NC);
    }
}

template <int D, bool BF16, bool SPLIT>
hipError_t launch_k(const AttnArgs &a)
{
    switch (a.k) {
    case 1: return launch_typed<D, BF16, 1, SPLIT>(a);
    case 2: return launch_typed<D, BF16, 2, SPLIT>(a);
    case 3: return launch_typed<D, BF16, 3, SPLIT>(a);
    case 4: return launch_typed<D, BF16, 4, SPLIT>(a);
    case 5: return launch_typed<D, BF16, 5, SPLIT>(a);
    case 6: return launch_typed<D, BF16, 6, SPLIT>(a);
    case 7: return launch_typed<D, BF16, 7, SPLIT>(a);
    case 8: return launch_typed<D, BF16, 8, SPLIT>(a);
    default: return hipErrorInvalidValue;
    }
}

template <bool BF16, bool SPLIT>
hipError_t launch_d(const AttnArgs &a)
{
    switch (a.D) {
    case 16: return launch_k<16, BF16, SPLIT>(a);
    case 32: return launch_k<32, BF16, SPLIT>(a);
    case 64: return launch_k<64, BF16, SPLIT>(a);
    case 128: return launch_k<128, BF16, SPLIT>(a);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

namespace {
std::atomic<int> g_path_override{0};
}  // namespace

hipError_t set_attn_trace(unsigned long long *buf, unsigned int cap) {
#if FS_TRACE
    const trace::Target t{buf, cap};
    return hipMemcpyToSymbol(HIP_SYMBOL(g_trace), &t, sizeof(t));
#else
    (void)buf;
    (void)cap;
    return hipErrorNotSupported;
#endif
}

AttnPath set_attn_path_override(AttnPath p) {
    return static_cast<AttnPath>(g_path_override.exchange(static_cast<int>(p), std::memory_order_relaxed));
}

AttnPath choose_attn_path(int n_bh, int jobs_max) {
    const AttnPath forced = static_cast<AttnPath>(g_path_override.load(std::memory_order_relaxed));
    if (forced != AttnPath::kAuto) return forced;
    // Measured on MI355X (bf16, D = 64, k = 4 or 5; 192 to 5120 rows of up to
    // 1024 keys): an 8-wave workgroup per row (two jobs in flight) is the
    // fastest from 256 rows up (BART-shaped 512 rows: 18.6 us against 19.5
    // for 4 waves; 5120 rows: 128 us against 134); with fewer rows than CUs
    // a 16-wave workgroup per row uses the idle CUs' share of the row's
    // jobs (192 rows of the split cache: 12.9 us against 13.9).  Rows of a
    // single job take 4 waves, and only a few long rows are split across
    // workgroups, whose merge costs a round trip through memory.
    if (jobs_max <= 1) return AttnPath::kWhole1;
    if (jobs_max <= 2) return AttnPath::kWhole2;
    if (n_bh < kWhole2MinRows) return AttnPath::kSplit;
    if (n_bh < kCus) return AttnPath::kWhole4;
    return AttnPath::kWhole2;
}

int cross_attn_chunk_keys(int D, int esize) {
    // kWaves * kIt rows of 64/(lanes per row) = 4 * 8 * 64 * 16 / (D * esize)
    return kWaves * kIt * kWave * 16 / (D * esize);
}

size_t cross_attn_workspace_floats(int B, int k, int H, int S, int D, int esize, bool split) {
    const int C = cross_attn_chunk_keys(D, esize);
    // one record per tile of the row (kWaves tiles per chunk), plus the
    // generated-token record of the split cache
    const size_t NT = (size_t)std::max(1, (S + C - 1) / C) * kWaves + (split ? 1 : 0);
    const size_t n_bh = (size_t)B * H;
    const size_t part = n_bh * NT * (size_t)k * (size_t)(D + 2);
    return 2 * (part + n_bh);  // 64-bit words: the partial records, then one counter per row
}

hipError_t launch_cross_attn(const void *q, const void *K, const void *V, const int32_t *src_len,
                             void *out, int B, int k, int H, int S, int D, bool bf16,
                             float *workspace, unsigned long long epoch, hipStream_t stream,
                             AttnPath path, const NgramRows *ngram)
{
    AttnArgs a{q, K, V, src_len, out, B, k, H, S, D, nullptr, nullptr, 0, 0, nullptr, 0, workspace, epoch, stream,
               NgramJob{nullptr, nullptr, 0, 0, 0, 0, 0, 0}, path};
    if (ngram)
        a.ng = NgramJob{ngram->tokens, ngram->logits, ngram->ld, ngram->t, ngram->n - 1, ngram->V, ngram->rows, 0};
    return bf16 ? launch_d<true, false>(a) : launch_d<false, false>(a);
}

hipError_t launch_prefix_attn(const void *q, const void *Kp, const void *Vp, const int32_t *prefix_len,
                              const void *Kt, const void *Vt, int T, int t, const int32_t *anc, int ld_anc,
                              void *out, int B, int k, int H, int N, int D, bool bf16, float *workspace,
                              unsigned long long epoch, hipStream_t stream, AttnPath path)
{
    const AttnArgs a{q, Kp, Vp, prefix_len, out, B, k, H, N, D, Kt, Vt, T, t, anc, ld_anc, workspace, epoch, stream,
                     NgramJob{nullptr, nullptr, 0, 0, 0, 0, 0, 0}, path};
    return bf16 ? launch_d<true, true>(a) : launch_d<false, true>(a);
}

}  // namespace fs
