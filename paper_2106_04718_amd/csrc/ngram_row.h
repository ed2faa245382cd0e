// No-repeat-n-gram blocking of one hypothesis row by one wavefront, with n
// known only at run time (Section 4.2, Algorithm 1; the rule of
// fs_ngram_block).  The fused decode step runs it in workgroups of the
// attention grid, so the row scan needs no launch of its own.
//
// For n - 1 < 64 the row costs one memory round trip: lane l loads history
// positions l, l + 64, ... and window j = lane + 64 m takes the tokens that
// follow its first one from the next lanes (ds_bpermute across the wave,
// wrapping into the next 64 positions); the last n - 1 tokens are read with
// wave-uniform loads.  Longer n-grams compare against memory directly.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace fs {

// Value that lane (lane + c) holds in the 128-lane concatenation [lo | hi]
// (0 < c < 64).
__device__ __forceinline__ int32_t ngram_following(int32_t lo, int32_t hi, int lane, int c) {
    const int src = ((lane + c) & 63) << 2;
    const int32_t a = __builtin_amdgcn_ds_bpermute(src, lo);
    const int32_t b = __builtin_amdgcn_ds_bpermute(src, hi);
    return lane + c < 64 ? a : b;
}

// Bans of row x[0 .. t-1] written into lg[0 .. V-1]; nm1 = n - 1 >= 0.
// Every lane of the wave must call it with the same arguments.
__device__ __forceinline__ void ngram_wave_row(const int32_t *__restrict__ x, int t, int nm1,
                                               float *__restrict__ lg, int V, int lane) {
    const int nwin = t - nm1;  // windows j = 0 .. t-n
    if (nwin <= 0) return;
    if (nm1 < 64) {
        constexpr int kM = 4;  // 64-position slices per pass, loaded together
        for (int base = 0; base < nwin; base += kM * 64) {
            int32_t s[kM + 1];
#pragma unroll
            for (int m = 0; m <= kM; ++m) {
                const int pos = base + m * 64 + lane;
                s[m] = pos < t ? x[pos] : 0;
            }
#pragma unroll
            for (int m = 0; m < kM; ++m) {
                const int j = base + m * 64 + lane;
                int diff = 0;
                int32_t v = s[m];
                for (int c = 0; c < nm1; ++c) {
                    diff |= v ^ x[t - nm1 + c];
                    v = ngram_following(s[m], s[m + 1], lane, c + 1);
                }
                if (j < nwin && diff == 0 && (uint32_t)v < (uint32_t)V) lg[v] = -INFINITY;
            }
        }
    } else {
        for (int j = lane; j < nwin; j += 64) {
            int diff = 0;
            for (int c = 0; c < nm1; ++c) diff |= x[j + c] ^ x[t - nm1 + c];
            const int32_t v = x[j + nm1];
            if (diff == 0 && (uint32_t)v < (uint32_t)V) lg[v] = -INFINITY;
        }
    }
}

// The n-gram part of a fused decode step: `rows` hypotheses, one wave each,
// handled by the first `blocks` workgroups of the launch (waves_per_block
// rows per workgroup).  blocks == 0: no n-gram part.
struct NgramJob {
    const int32_t *tokens;
    float *logits;
    int ld, t, nm1, V, rows, blocks;
};

// Workgroup g < job.blocks scans rows g * waves_per_block + wave.
__device__ __forceinline__ void ngram_job_block(const NgramJob &job, int g, int waves_per_block) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int lane = threadIdx.x & 63;
    const int r = g * waves_per_block + wave;
    if (r >= job.rows) return;
    ngram_wave_row(job.tokens + (size_t)r * job.ld, job.t, job.nm1, job.logits + (size_t)r * job.V, job.V, lane);
}

}  // namespace fs
