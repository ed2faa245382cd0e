// Workgroup timelines of trace builds (compiled with FS_TRACE=1; in every
// other build each call below is empty and the kernels are unchanged).
//
// A traced kernel's workgroup g writes up to 8 64-bit words at
// buffer[8 g .. 8 g + 7] -- clock stamps (s_memrealtime, 100 MHz), its
// hardware ids and a few counts; what each word holds is given where the
// kernel stamps it.  Workgroups at or past the buffer's capacity write
// nothing.  The buffer is set per translation unit (trace_set_* in
// launch.h) and read back by the caller after the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#ifndef FS_TRACE
#define FS_TRACE 0
#endif

namespace fs {
namespace trace {

struct Target {
    unsigned long long *buf;
    unsigned int cap;   // workgroups
};

#if FS_TRACE
// this workgroup's words, or null (no buffer, or past its capacity); only
// the first thread of the workgroup writes
__device__ __forceinline__ unsigned long long *slot(const Target &t) {
    return (t.buf && threadIdx.x == 0 && blockIdx.x < t.cap) ? t.buf + (size_t)blockIdx.x * 8 : nullptr;
}
__device__ __forceinline__ void stamp(unsigned long long *s, int i) {
    if (s) s[i] = __builtin_amdgcn_s_memrealtime();
}
__device__ __forceinline__ void put(unsigned long long *s, int i, unsigned long long v) {
    if (s) s[i] = v;
}
// HW_ID (compute unit, SIMD, shader array and engine) in the low 32 bits,
// XCC_ID in the high 32
__device__ __forceinline__ unsigned long long where() {
    const unsigned hw = __builtin_amdgcn_s_getreg((4 << 0) | (0 << 6) | (31 << 11));
    const unsigned xcc = __builtin_amdgcn_s_getreg((20 << 0) | (0 << 6) | (31 << 11));
    return ((unsigned long long)xcc << 32) | hw;
}
#else
__device__ __forceinline__ unsigned long long *slot(const Target &) { return nullptr; }
__device__ __forceinline__ void stamp(unsigned long long *, int) {}
__device__ __forceinline__ void put(unsigned long long *, int, unsigned long long) {}
__device__ __forceinline__ unsigned long long where() { return 0; }
#endif

}  // namespace trace
}  // namespace fs
