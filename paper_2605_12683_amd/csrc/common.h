// Internal helpers shared by the libdeer translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/deer.h"

typedef float v4f __attribute__((ext_vector_type(4)));

namespace deer {

// ---- host-side error plumbing --------------------------------------------------------
void set_error(const char *fmt, ...);
int hip_fail(hipError_t e, const char *what);

#define DEER_HIP(call)                                                 \
    do {                                                               \
        hipError_t _e = (call);                                        \
        if (_e != hipSuccess) return ::deer::hip_fail(_e, #call);      \
    } while (0)

#define DEER_LAUNCH_CHECK(what)                                        \
    do {                                                               \
        hipError_t _e = hipGetLastError();                             \
        if (_e != hipSuccess) return ::deer::hip_fail(_e, what);       \
    } while (0)

// ---- optional per-kernel timing (HIP events on the launching stream) ----------------------
// Off unless deer_timing_enable(1) was called; then every launch site brackets its kernel
// with two events taken from a pool.
bool timing_on();
void timing_mark(const char *name, hipStream_t st, bool start);

// While one of these lives on a thread, no launch of that thread is timed (no events are made).
void timing_suppress(bool on);
bool timing_suppressed();
struct TimingSuppress {
    bool prev;
    TimingSuppress() : prev(timing_suppressed()) { timing_suppress(true); }
    ~TimingSuppress() { timing_suppress(prev); }
};

struct KTimer {
    const char *name;
    hipStream_t st;
    bool on;
    KTimer(const char *n, hipStream_t s) : name(n), st(s), on(timing_on()) {
        if (on) timing_mark(name, st, true);
    }
    ~KTimer() {
        if (on) timing_mark(name, st, false);
    }
};

// ---- device helpers ---------------------------------------------------------------------

// 16x16x4 fp32 MFMA: acc[16x16] += A[16x4] * B[4x16].  Lane l = 16*g + c holds
// A[c][g], B[g][c] and acc[4*g + r][c] in element r of the returned vector.
__device__ __forceinline__ v4f mfma16x16x4(float a, float b, v4f acc) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
}

// all-ones if bit `sh` of w is set, else zero (sign-extended one-bit field)
__device__ __forceinline__ float select_bit(uint32_t w, int sh, float v) {
    int m = __builtin_amdgcn_sbfe((int)w, sh, 1);
    return __int_as_float(__float_as_int(v) & m);
}

// |v| as ordered bits: NaN (any sign) compares above +Inf, so an unsigned max keeps NaN.
__device__ __forceinline__ uint32_t abs_bits(float v) {
    return (uint32_t)__float_as_int(v) & 0x7fffffffu;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = (uint32_t)__shfl_xor((int)v, off, 64);
        v = v > o ? v : o;
    }
    return v;
}

// Buffer resource with a wave-uniform base: an access adds a per-lane byte offset (VGPR) and a
// wave-uniform byte offset (SGPR).  A lane offset of 2^31 or more is outside the resource: a
// load from it returns zero and a store to it is dropped.
constexpr uint32_t kOffLane = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t wave_rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ uint32_t bload_u(__amdgpu_buffer_rsrc_t rs, uint32_t voff, int soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(rs, (int)voff, soff, 0);
}
__device__ __forceinline__ float bload(__amdgpu_buffer_rsrc_t rs, uint32_t voff, int soff) {
    return __uint_as_float(bload_u(rs, voff, soff));
}
__device__ __forceinline__ void bstore_u(__amdgpu_buffer_rsrc_t rs, uint32_t v, uint32_t voff, int soff) {
    __builtin_amdgcn_raw_buffer_store_b32(v, rs, (int)voff, soff, 0);
}
// The same over `bytes` bytes from base (bytes < 2^31): an access at or past the end reads zero
// and a store there is dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t bounded_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// forced input of step s (array index) for latent i:
//   s == 0: z0 (or [x_0; 0] when z0 is null);  s >= 1: fl(fl(p*z_{s-1}) + fl(a*zbar_s))
// The two iterate buffers of the safeguarded Newton loop: sequence b's current iterate is in
// zalt when zsel[b] is set, else in z, and an update is written to the other buffer.  With
// zsel null and zalt == z the update is applied in place.
__device__ __forceinline__ const float *cur_iter(const float *z, const float *zalt, const int *zsel, int b) {
    return (zsel && zsel[b]) ? zalt : z;
}
__device__ __forceinline__ float *next_iter(float *z, float *zalt, const int *zsel, int b) {
    return (zsel && zsel[b]) ? z : zalt;
}

// (sequence, step) of the rows row0 + rr of a [B, T] row space: the first row's pair from one
// division per tile, the others by carrying over sequence ends (rr small), instead of a 64-bit
// division per row
struct RowBase {
    int b0, s0;
};
__device__ __forceinline__ RowBase row_base(long row0, int T) {
    const long b = row0 / T;
    return {(int)b, (int)(row0 - b * T)};
}
__device__ __forceinline__ void row_at(RowBase rb, int rr, int T, int &b, int &s) {
    s = rb.s0 + rr;
    b = rb.b0;
    while (s >= T) {
        s -= T;
        ++b;
    }
}

// Workgroup barrier that orders LDS only: unlike __syncthreads it does not wait for
// outstanding global loads, so loads issued ahead (prefetch) stay in flight across it.  For
// kernels whose threads exchange data through LDS alone.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The same for data exchanged through LDS between the lanes of one wave only: the LDS writes
// complete before the reads after it, and no other wave is waited for.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float forced_state(const float *__restrict__ x, const float *__restrict__ z0,
                                              const float *__restrict__ z, int b, int s, int i, int T, int M,
                                              int N, float alpha, int tw = 0) {
    if (s == 0) {
        if (z0) return z0[(size_t)b * M + i];
        return i < N ? x[(size_t)b * (T + 1) * N + i] : 0.0f;
    }
    float zp = z[((size_t)b * T + (s - 1)) * M + i];
    if (i >= N) return zp;
    float zb = x[((size_t)b * (T + 1) + s) * N + i];
    if (s <= tw) return zb;   // latent warm-up: alpha_s = 1 for s = 1..tw
    float p = __fsub_rn(1.0f, alpha);
    return __fadd_rn(__fmul_rn(p, zp), __fmul_rn(alpha, zb));
}

}  // namespace deer
