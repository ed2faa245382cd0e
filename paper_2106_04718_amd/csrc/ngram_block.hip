// No-repeat-n-gram blocking on the GPU, for gfx950.
//
// The operation is Algorithm 1 of the paper (Section 4.2): for hypothesis
// row r with history x[0..t-1], every window start j in [0, t-n] whose n-1
// tokens x[j..j+n-2] equal the row's last n-1 tokens bans the token that
// followed, x[j+n-1], by writing -inf into logits[r, x[j+n-1]].
//
// The paper launches one block per row and one thread per window, with the
// row staged in shared memory.  Here one wavefront handles one row, and the
// kernel is built around a single memory round trip:
//   - all the row's tokens are loaded at once, lane l holding positions
//     l, l+64, ... (coalesced), and the last n-1 tokens with wave-uniform
//     loads issued alongside;
//   - window j = lane + 64m takes its n tokens from its own register and
//     from lanes l+1 .. l+n-1 (ds_bpermute across the wave, wrapping into
//     the next 64 positions), and compares the (n-1)-gram in registers;
//   - matching lanes scatter -inf; the logits are never read.
// Several windows that ban the same id write the same bits, so no atomics
// are needed.
#include <math.h>

#include "launch.h"

namespace fs {
namespace {

constexpr int kWave = 64;

// Value that lane (lane + c) holds in the 128-lane concatenation [lo | hi]
// (0 < c < 64): the window tokens that follow this lane's position.
__device__ __forceinline__ int32_t following(int32_t lo, int32_t hi, int lane, int c) {
    const int src = ((lane + c) & (kWave - 1)) << 2;
    const int32_t a = __builtin_amdgcn_ds_bpermute(src, lo);
    const int32_t b = __builtin_amdgcn_ds_bpermute(src, hi);
    return lane + c < kWave ? a : b;
}

// NM1 = n - 1 known at compile time (0..7).
template <int NM1>
__global__ __launch_bounds__(kWave) void ngram_block_fixed(
    const int32_t *__restrict__ tokens, int ld, int t, float *__restrict__ logits, int V)
{
    constexpr int kM = 4;  // 64-position slices per pass (all loaded together)
    const int row = blockIdx.x;
    const int lane = threadIdx.x;
    const int32_t *x = tokens + (size_t)row * ld;
    float *lg = logits + (size_t)row * V;
    const int nwin = t - NM1;  // windows j = 0 .. t-n
    if (nwin <= 0) return;

    int32_t suf[NM1 > 0 ? NM1 : 1];
#pragma unroll
    for (int c = 0; c < NM1; ++c) suf[c] = x[t - NM1 + c];

    for (int base = 0; base < nwin; base += kM * kWave) {
        int32_t s[kM + 1];
#pragma unroll
        for (int m = 0; m <= kM; ++m) {
            const int pos = base + m * kWave + lane;
            s[m] = pos < t ? x[pos] : 0;
        }
#pragma unroll
        for (int m = 0; m < kM; ++m) {
            const int j = base + m * kWave + lane;
            int diff = 0;
            int32_t v = s[m];
#pragma unroll
            for (int c = 0; c < NM1; ++c) {
                diff |= v ^ suf[c];
                v = following(s[m], s[m + 1], lane, c + 1);
            }
            if (j < nwin && diff == 0 && (uint32_t)v < (uint32_t)V) lg[v] = -INFINITY;
        }
    }
}

// Any n >= 1: the suffix is re-read from memory (L1 hits) per comparison.
__global__ __launch_bounds__(kWave) void ngram_block_any(
    const int32_t *__restrict__ tokens, int ld, int t, int n, float *__restrict__ logits, int V)
{
    const int row = blockIdx.x;
    const int lane = threadIdx.x;
    const int32_t *x = tokens + (size_t)row * ld;
    float *lg = logits + (size_t)row * V;
    const int nm1 = n - 1;
    const int nwin = t - nm1;
    for (int j = lane; j < nwin; j += kWave) {
        int diff = 0;
        for (int c = 0; c < nm1; ++c) diff |= x[j + c] ^ x[t - nm1 + c];
        const int32_t v = x[j + nm1];
        if (diff == 0 && (uint32_t)v < (uint32_t)V) lg[v] = -INFINITY;
    }
}

template <int NM1>
void launch_fixed(const int32_t *tokens, int ld, int rows, int t, float *logits, int V,
                  hipStream_t stream)
{
    hipLaunchKernelGGL(ngram_block_fixed<NM1>, dim3((unsigned)rows), dim3(kWave), 0, stream,
                       tokens, ld, t, logits, V);
}

}  // namespace

hipError_t launch_ngram_block(const int32_t *tokens, int ld_tokens, int rows, int t, int n,
                              float *logits, int V, hipStream_t stream)
{
    switch (n - 1) {
    case 0: launch_fixed<0>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 1: launch_fixed<1>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 2: launch_fixed<2>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 3: launch_fixed<3>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 4: launch_fixed<4>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 5: launch_fixed<5>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 6: launch_fixed<6>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    case 7: launch_fixed<7>(tokens, ld_tokens, rows, t, logits, V, stream); break;
    default:
        hipLaunchKernelGGL(ngram_block_any, dim3((unsigned)rows), dim3(kWave), 0, stream,
                           tokens, ld_tokens, t, n, logits, V);
        break;
    }
    return hipGetLastError();
}

}  // namespace fs
