// Products of a 16 x 16 matrix with a vector held by the 16 lanes of a wave row, by DPP row
// rotations (internal to libdeer, not part of the ABI).
#pragma once

#include "common.h"

namespace deer {

// lane l of each 16-lane row receives v from lane row_src(l, K) of the same row
template <int K>
__device__ __forceinline__ int row_ror_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, 0x120 + K, 0xF, 0xF, true);
}

// source lane (within the row) of rotation k, k = 0..15
__device__ __forceinline__ void row_sources(int c, int (&src)[16]) {
    src[0] = c;
    src[1] = row_ror_i<1>(c);   src[2] = row_ror_i<2>(c);   src[3] = row_ror_i<3>(c);
    src[4] = row_ror_i<4>(c);   src[5] = row_ror_i<5>(c);   src[6] = row_ror_i<6>(c);
    src[7] = row_ror_i<7>(c);   src[8] = row_ror_i<8>(c);   src[9] = row_ror_i<9>(c);
    src[10] = row_ror_i<10>(c); src[11] = row_ror_i<11>(c); src[12] = row_ror_i<12>(c);
    src[13] = row_ror_i<13>(c); src[14] = row_ror_i<14>(c); src[15] = row_ror_i<15>(c);
}

// sum_k w[k] * v(row_src(lane, k)): with w[k] = W[i][row_src(i, k)] this is (W v)_i for the
// vector v held by the 16 lanes of the row.  One multiply-add with a DPP row rotation of v per
// term (the compiler does not fuse a rotation into v_fmac by itself); the leading s_nop covers
// the wait a DPP read needs after a VALU write of v.  All 64 lanes must be active.
#define DEER_RR(k) " row_ror:" #k " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
__device__ __forceinline__ float row16_dot(const float (&w)[16], float v) {
    float a0, a1;
    asm volatile(
        "s_nop 1\n"
        "v_mul_f32_e32 %0, %2, %3\n"
        "v_mul_f32_dpp %1, %2, %4" DEER_RR(1)
        "v_fmac_f32_dpp %0, %2, %5" DEER_RR(2)
        "v_fmac_f32_dpp %1, %2, %6" DEER_RR(3)
        "v_fmac_f32_dpp %0, %2, %7" DEER_RR(4)
        "v_fmac_f32_dpp %1, %2, %8" DEER_RR(5)
        "v_fmac_f32_dpp %0, %2, %9" DEER_RR(6)
        "v_fmac_f32_dpp %1, %2, %10" DEER_RR(7)
        "v_fmac_f32_dpp %0, %2, %11" DEER_RR(8)
        "v_fmac_f32_dpp %1, %2, %12" DEER_RR(9)
        "v_fmac_f32_dpp %0, %2, %13" DEER_RR(10)
        "v_fmac_f32_dpp %1, %2, %14" DEER_RR(11)
        "v_fmac_f32_dpp %0, %2, %15" DEER_RR(12)
        "v_fmac_f32_dpp %1, %2, %16" DEER_RR(13)
        "v_fmac_f32_dpp %0, %2, %17" DEER_RR(14)
        "v_fmac_f32_dpp %1, %2, %18" DEER_RR(15)
        : "=&v"(a0), "=&v"(a1)
        : "v"(v), "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]), "v"(w[8]),
          "v"(w[9]), "v"(w[10]), "v"(w[11]), "v"(w[12]), "v"(w[13]), "v"(w[14]), "v"(w[15]));
    return a0 + a1;
}

// two independent row products W v0, W v1 (each summed exactly as row16_dot), interleaved so
// that dependent multiply-adds are four instructions apart
__device__ __forceinline__ void row16_dot2(const float (&w)[16], float v0, float v1, float &r0, float &r1) {
    float a0, a1, b0, b1;
    asm volatile(
        "s_nop 1\n"
        "v_mul_f32_e32 %0, %4, %6\n"
        "v_mul_f32_e32 %2, %5, %6\n"
        "v_mul_f32_dpp %1, %4, %7" DEER_RR(1)
        "v_mul_f32_dpp %3, %5, %7" DEER_RR(1)
        "v_fmac_f32_dpp %0, %4, %8" DEER_RR(2)
        "v_fmac_f32_dpp %2, %5, %8" DEER_RR(2)
        "v_fmac_f32_dpp %1, %4, %9" DEER_RR(3)
        "v_fmac_f32_dpp %3, %5, %9" DEER_RR(3)
        "v_fmac_f32_dpp %0, %4, %10" DEER_RR(4)
        "v_fmac_f32_dpp %2, %5, %10" DEER_RR(4)
        "v_fmac_f32_dpp %1, %4, %11" DEER_RR(5)
        "v_fmac_f32_dpp %3, %5, %11" DEER_RR(5)
        "v_fmac_f32_dpp %0, %4, %12" DEER_RR(6)
        "v_fmac_f32_dpp %2, %5, %12" DEER_RR(6)
        "v_fmac_f32_dpp %1, %4, %13" DEER_RR(7)
        "v_fmac_f32_dpp %3, %5, %13" DEER_RR(7)
        "v_fmac_f32_dpp %0, %4, %14" DEER_RR(8)
        "v_fmac_f32_dpp %2, %5, %14" DEER_RR(8)
        "v_fmac_f32_dpp %1, %4, %15" DEER_RR(9)
        "v_fmac_f32_dpp %3, %5, %15" DEER_RR(9)
        "v_fmac_f32_dpp %0, %4, %16" DEER_RR(10)
        "v_fmac_f32_dpp %2, %5, %16" DEER_RR(10)
        "v_fmac_f32_dpp %1, %4, %17" DEER_RR(11)
        "v_fmac_f32_dpp %3, %5, %17" DEER_RR(11)
        "v_fmac_f32_dpp %0, %4, %18" DEER_RR(12)
        "v_fmac_f32_dpp %2, %5, %18" DEER_RR(12)
        "v_fmac_f32_dpp %1, %4, %19" DEER_RR(13)
        "v_fmac_f32_dpp %3, %5, %19" DEER_RR(13)
        "v_fmac_f32_dpp %0, %4, %20" DEER_RR(14)
        "v_fmac_f32_dpp %2, %5, %20" DEER_RR(14)
        "v_fmac_f32_dpp %1, %4, %21" DEER_RR(15)
        "v_fmac_f32_dpp %3, %5, %21" DEER_RR(15)
        : "=&v"(a0), "=&v"(a1), "=&v"(b0), "=&v"(b1)
        : "v"(v0), "v"(v1), "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]),
          "v"(w[8]), "v"(w[9]), "v"(w[10]), "v"(w[11]), "v"(w[12]), "v"(w[13]), "v"(w[14]), "v"(w[15]));
    r0 = a0 + a1;
    r1 = b0 + b1;
}
#undef DEER_RR

}  // namespace deer
