// Encoder-decoder cross-attention over a de-duplicated K/V cache, for gfx950.
//
// The operation is Eq. 4 of the paper (Appendix B): the k beam queries of
// source b read the one copy K[b], V[b] of that source's encoder keys and
// values, and each computes softmax(q K^T / sqrt(D)) V over the valid keys
// j < src_len[b].  Per head it is a GEMV-like contraction with k query rows,
// so it is bound by HBM bandwidth (about k flop per byte of K/V); the design
// goal is to read every valid K/V byte exactly once, coalesced, and to keep
// the VALU work per byte small enough to stay under the memory time.
//
// Work split (split-KV):
//   kernel 1, one workgroup per (source b, head h, chunk c of C keys):
//     Each of the 4 waves owns one tile of 64 consecutive keys of the chunk.
//     QK^T:  lane j of the wave holds key j's whole row and forms the k
//            scores itself (no cross-lane reduction); the k queries sit in
//            LDS and are read as broadcasts.
//     softmax: the tile's maximum and sum per beam are wave reductions, so
//            every exponential is taken once per (key, beam).
//     PV:    the weights go through LDS to a coalesced layout in which a
//            group of lanes shares one V row (16 bytes per lane) and each lane
//            accumulates k x (its 16 bytes of dims) in fp32.
//     The four tiles are merged in fixed order and the chunk's partial
//     (max, sum, unnormalised output) is written to the workspace.
//   kernel 2, one workgroup per (b, h): merges the chunks of the source in
//     order by log-sum-exp, normalises, rounds and stores.
// Rows j >= src_len[b] are never read.  The chunk size depends only on the
// row size, and each beam's arithmetic is the same whatever k is, so the
// output bits do not depend on k, B or the beam's position.
#include <math.h>

#include "launch.h"

namespace fs {
namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWave * kWaves;
constexpr int kTile = kWave;  // keys per wave tile: one key per lane

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

template <bool BF16>
struct Elem {
    static constexpr int size = BF16 ? 2 : 4;
    static constexpr int per16 = 16 / size;  // elements in 16 bytes
};

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

// Cross-lane moves.  DPP quad_perm/row mirrors stay inside a row of 16
// lanes; ds_swizzle covers the 32-lane halves and ds_bpermute the rest.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;  // lane i <-> 7-i within 8 lanes
constexpr int kRowMirror = 0x140;      // lane i <-> 15-i within 16 lanes

__device__ __forceinline__ float swz_xor16(float x) {
    // BitMode swizzle inside 32 lanes: and 0x1f, or 0, xor 0x10.
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
}

__device__ __forceinline__ float shfl_xor(float x, int mask);

// Butterfly all-reduce over the 64 lanes; every lane gets the same value.
// Each step combines (own, partner) with a commutative operation, so the
// two lanes of a pair compute bit-identical results.
__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp<kQuadXor1>(x));
    x = fmaxf(x, dpp<kQuadXor2>(x));
    x = fmaxf(x, dpp<kRowHalfMirror>(x));
    x = fmaxf(x, dpp<kRowMirror>(x));
    x = fmaxf(x, swz_xor16(x));
    x = fmaxf(x, shfl_xor(x, 32));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp<kQuadXor1>(x);
    x += dpp<kQuadXor2>(x);
    x += dpp<kRowHalfMirror>(x);
    x += dpp<kRowMirror>(x);
    x += swz_xor16(x);
    x += shfl_xor(x, 32);
    return x;
}

__device__ __forceinline__ float shfl_xor(float x, int mask) {
    const int lane = __lane_id();
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ mask) << 2,
                                                                  __builtin_bit_cast(int, x)));
}

// Sum over the lanes that share (lane % Group): the lane groups of the PV
// layout hold partial sums of the same dims for different rows.
template <int Group>
__device__ __forceinline__ float sum_across_groups(float x) {
#pragma unroll
    for (int mask = Group; mask < kWave; mask <<= 1) x += shfl_xor(x, mask);
    return x;
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

template <int D, bool BF16, int KB>
struct Cfg {
    static constexpr int kEpl = Elem<BF16>::per16;  // elements per 16-byte slice
    static constexpr int kSlices = D / kEpl;        // 16-byte slices per row
    static constexpr int kLpr = kSlices;            // PV: lanes sharing one V row
    static constexpr int kRpi = kWave / kLpr;       // PV: rows per wave instruction
    static_assert(kSlices >= 2 && kSlices <= 32, "row must be 32..512 bytes");
};

// Kernel 1: one workgroup per (b, h, chunk).  Chunk c covers keys
// [c*C, c*C + C) with C = kWaves * kTile * tiles_per_wave.
template <int D, bool BF16, int KB>
__global__ __launch_bounds__(kBlock) void cross_attn_chunks(
    const uint4 *__restrict__ q, const uint4 *__restrict__ K, const uint4 *__restrict__ V,
    const int32_t *__restrict__ src_len, float *__restrict__ part,
    int H, int S, int C, int NC, float scale_log2)
{
    using CF = Cfg<D, BF16, KB>;
    constexpr int kS = CF::kSlices;
    constexpr int kEpl = CF::kEpl;
    constexpr int kLpr = CF::kLpr;
    constexpr int kRpi = CF::kRpi;

    __shared__ uint4 q_lds[KB * kS];
    __shared__ float p_lds[kWaves][kTile][KB];
    __shared__ float m_lds[kWaves][KB], l_lds[kWaves][KB];
    __shared__ float a_lds[kWaves][KB][D];

    const int bh = blockIdx.x / NC;
    const int c = blockIdx.x - bh * NC;
    const int b = bh / H;
    const int h = bh - b * H;
    const int L = min(max(src_len[b], 0), S);
    const int j0 = c * C;
    if (j0 >= L) return;  // whole chunk is padding: never read
    const int j1 = min(j0 + C, L);

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = tid / kWave;

    // k queries of (b, h): q[b, i, h, :] for i < KB
    for (int x = tid; x < KB * kS; x += kBlock) {
        const int i = x / kS, s = x - i * kS;
        q_lds[x] = q[((size_t)(b * KB + i) * H + h) * kS + s];
    }
    __syncthreads();

    const uint4 *Kbh = K + (size_t)bh * S * kS;
    const uint4 *Vbh = V + (size_t)bh * S * kS;

    const int sub = lane % kLpr;  // PV: this lane's slice of the row
    const int grp = lane / kLpr;  // PV: this lane's row within an instruction

    float m[KB], l[KB], acc[KB][kEpl];
#pragma unroll
    for (int i = 0; i < KB; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
#pragma unroll
        for (int e = 0; e < kEpl; ++e) acc[i][e] = 0.f;
    }

    // Every wave runs the same number of iterations (the loop holds
    // barriers); a wave whose tile lies past j1 sees only invalid keys.
    for (int tb = j0; tb < j1; tb += kWaves * kTile) {
        const int t0 = tb + w * kTile;
        // ---- QK^T: lane owns key t0 + lane -------------------------------
        const int j = t0 + lane;
        const bool valid = j < j1;
        uint4 kr[kS];
#pragma unroll
        for (int s = 0; s < kS; ++s) kr[s] = make_uint4(0, 0, 0, 0);
        if (valid) {
#pragma unroll
            for (int s = 0; s < kS; ++s) kr[s] = Kbh[(size_t)j * kS + s];
        }
        // V slices for the PV layout: instruction u covers rows u*kRpi + grp
        uint4 vr[kTile / kRpi];
#pragma unroll
        for (int u = 0; u < kTile / kRpi; ++u) {
            const int jv = t0 + u * kRpi + grp;
            vr[u] = make_uint4(0, 0, 0, 0);
            if (jv < j1) vr[u] = Vbh[(size_t)jv * kS + sub];
        }

        float s_[KB];
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            float d = 0.f;
#pragma unroll
            for (int s = 0; s < kS; ++s) d = dot16<BF16>(q_lds[i * kS + s], kr[s], d);
            s_[i] = valid ? d * scale_log2 : -INFINITY;
        }

        // ---- softmax over the tile, once per (key, beam) -----------------
        float p[KB];
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            const float mt = wave_max(s_[i]);
            const float ms = (mt == -INFINITY) ? 0.f : mt;
            p[i] = __builtin_amdgcn_exp2f(s_[i] - ms);
            const float lt = wave_sum(p[i]);
            // fold the tile into the running state (wave-uniform m, l)
            const float mx = fmaxf(m[i], mt);
            const float mxs = (mx == -INFINITY) ? 0.f : mx;
            const float fo = __builtin_amdgcn_exp2f(m[i] - mxs);  // old state
            const float fn = __builtin_amdgcn_exp2f(mt - mxs);    // this tile
            l[i] = l[i] * fo + lt * fn;
#pragma unroll
            for (int e = 0; e < kEpl; ++e) acc[i][e] *= fo;
            m[i] = mx;
            p[i] *= fn;
        }
#pragma unroll
        for (int i = 0; i < KB; ++i) p_lds[w][lane][i] = p[i];
        __syncthreads();

        // ---- PV: coalesced rows, weights broadcast from LDS ---------------
#pragma unroll
        for (int u = 0; u < kTile / kRpi; ++u) {
            const int r = u * kRpi + grp;
            float vf[kEpl];
            unpack16<BF16>(vr[u], vf);
#pragma unroll
            for (int i = 0; i < KB; ++i) {
                const float pw = p_lds[w][r][i];
#pragma unroll
                for (int e = 0; e < kEpl; ++e) acc[i][e] = fmaf(pw, vf[e], acc[i][e]);
            }
        }
        __syncthreads();
    }

    // ---- merge: lane groups of the wave (same m, l), then the 4 waves ----
#pragma unroll
    for (int i = 0; i < KB; ++i) {
#pragma unroll
        for (int e = 0; e < kEpl; ++e) acc[i][e] = sum_across_groups<kLpr>(acc[i][e]);
    }
    if (lane < kLpr) {
#pragma unroll
        for (int i = 0; i < KB; ++i) {
#pragma unroll
            for (int e = 0; e < kEpl; ++e) a_lds[w][i][sub * kEpl + e] = acc[i][e];
        }
    }
    if (lane == 0) {
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            m_lds[w][i] = m[i];
            l_lds[w][i] = l[i];
        }
    }
    __syncthreads();

    // partial record of (b, h, c): acc[KB][D], then m[KB], then l[KB]
    float *rec = part + ((size_t)bh * NC + c) * (size_t)(KB * (D + 2));
    for (int x = tid; x < KB * D; x += kBlock) {
        const int i = x / D, d = x - i * D;
        float mm = m_lds[0][i], ll = l_lds[0][i], aa = a_lds[0][i][d];
#pragma unroll
        for (int ww = 1; ww < kWaves; ++ww) merge_state(mm, ll, aa, m_lds[ww][i], l_lds[ww][i], a_lds[ww][i][d]);
        rec[x] = aa;
        if (d == 0) {
            rec[KB * D + i] = mm;
            rec[KB * D + KB + i] = ll;
        }
    }
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Kernel 2: one workgroup per (b, h); thread x = (beam i, dim d).
template <bool BF16, int KB>
__global__ __launch_bounds__(kBlock) void cross_attn_combine(
    const float *__restrict__ part, const int32_t *__restrict__ src_len, void *__restrict__ out,
    int H, int S, int D, int C, int NC)
{
    const int bh = blockIdx.x;
    const int b = bh / H;
    const int h = bh - b * H;
    const int L = min(max(src_len[b], 0), S);
    const int nc = (L + C - 1) / C;
    const size_t rs = (size_t)KB * (D + 2);
    for (int x = threadIdx.x; x < KB * D; x += blockDim.x) {
        const int i = x / D, d = x - i * D;
        float m = -INFINITY, l = 0.f, a = 0.f;
        for (int c = 0; c < nc; ++c) {
            const float *rec = part + ((size_t)bh * NC + c) * rs;
            merge_state(m, l, a, rec[KB * D + i], rec[KB * D + KB + i], rec[x]);
        }
        const float o = (nc == 0) ? 0.f : a / l;
        const size_t oi = ((size_t)(b * KB + i) * H + h) * D + d;
        if constexpr (BF16)
            static_cast<uint16_t *>(out)[oi] = f32_to_bf16_rne(o);
        else
            static_cast<float *>(out)[oi] = o;
    }
}

template <int D, bool BF16, int KB>
hipError_t launch_typed(const void *q, const void *K, const void *V, const int32_t *src_len,
                        void *out, int B, int H, int S, float *ws, hipStream_t stream)
{
    const int C = cross_attn_chunk_keys(D, Elem<BF16>::size);
    const int NC = (S + C - 1) / C;
    const double scale_log2 = 1.4426950408889634074 / sqrt((double)D);
    const long long nblk = (long long)B * H * NC;
    if (nblk > 0) {
        hipLaunchKernelGGL((cross_attn_chunks<D, BF16, KB>), dim3((unsigned)nblk), dim3(kBlock), 0,
                           stream, static_cast<const uint4 *>(q), static_cast<const uint4 *>(K),
                           static_cast<const uint4 *>(V), src_len, ws, H, S, C, NC,
                           (float)scale_log2);
    }
    hipLaunchKernelGGL((cross_attn_combine<BF16, KB>), dim3((unsigned)(B * H)), dim3(kBlock), 0,
                       stream, ws, src_len, out, H, S, D, C, NC);
    return hipGetLastError();
}

template <int D, bool BF16>
hipError_t launch_k(int k, const void *q, const void *K, const void *V, const int32_t *src_len,
                    void *out, int B, int H, int S, float *ws, hipStream_t stream)
{
    switch (k) {
    case 1: return launch_typed<D, BF16, 1>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 2: return launch_typed<D, BF16, 2>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 3: return launch_typed<D, BF16, 3>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 4: return launch_typed<D, BF16, 4>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 5: return launch_typed<D, BF16, 5>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 6: return launch_typed<D, BF16, 6>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 7: return launch_typed<D, BF16, 7>(q, K, V, src_len, out, B, H, S, ws, stream);
    case 8: return launch_typed<D, BF16, 8>(q, K, V, src_len, out, B, H, S, ws, stream);
    default: return hipErrorInvalidValue;
    }
}

template <bool BF16>
hipError_t launch_d(int D, int k, const void *q, const void *K, const void *V,
                    const int32_t *src_len, void *out, int B, int H, int S, float *ws,
                    hipStream_t stream)
{
    switch (D) {
    case 16: return launch_k<16, BF16>(k, q, K, V, src_len, out, B, H, S, ws, stream);
    case 32: return launch_k<32, BF16>(k, q, K, V, src_len, out, B, H, S, ws, stream);
    case 64: return launch_k<64, BF16>(k, q, K, V, src_len, out, B, H, S, ws, stream);
    case 128: return launch_k<128, BF16>(k, q, K, V, src_len, out, B, H, S, ws, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int cross_attn_chunk_keys(int D, int esize) {
    (void)D;
    (void)esize;
    return kWaves * kTile;  // one 64-key tile per wave
}

size_t cross_attn_workspace_floats(int B, int k, int H, int S, int D, int esize) {
    const int C = cross_attn_chunk_keys(D, esize);
    const size_t NC = (size_t)((S + C - 1) / C);
    return (size_t)B * H * NC * (size_t)k * (size_t)(D + 2);
}

hipError_t launch_cross_attn(const void *q, const void *K, const void *V, const int32_t *src_len,
                             void *out, int B, int k, int H, int S, int D, bool bf16,
                             float *workspace, hipStream_t stream)
{
    return bf16 ? launch_d<true>(D, k, q, K, V, src_len, out, B, H, S, workspace, stream)
                : launch_d<false>(D, k, q, K, V, src_len, out, B, H, S, workspace, stream);
}

}  // namespace fs
