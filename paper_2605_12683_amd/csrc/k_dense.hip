// Chunked associative scan over affine pairs (J_t, b_t) with the Jacobians stored in HBM
// ([B, T, M, M], row-major per step): the bare scan of deer_scan(DEER_SCAN_DENSE) and the
// linear solve of every shallow-PLRNN Newton update (scheduled-sampling appendix, the pair
// (A_t, b_t) and its composition; eq. GTF_DEER_update; eq. backward_recursion).
//
//   k_chunk_product_dense   per chunk: P_c = J_e ... J_s on the matrix cores (fp32 MFMA,
//                           A operand = J_t streamed from HBM, B operand = the accumulator
//                           itself, as in the vanilla kernel) and the chunk's local solution
//                           v_c from a zero carry (VALU)
//   k_fixup_dense           the chunk re-run from its carry: forward (Newton: z += Delta and
//                           max|Delta|; bare scan: y written) or reverse (y_{t-1} = J_t^T y_t + b)
// Carries across chunks use the shared k_carry kernel.
#include "common.h"
#include "launch.h"

namespace deer {

template <int MP>
struct DGeo {
    static constexpr int NCH = 64 / MP;
    static constexpr int NI = MP / 16;
    static constexpr int NS = MP / 4;
};

// J[row][col] of a step, zero outside M x M
__device__ __forceinline__ float jload(const float *__restrict__ Jp, int M, int row, int col) {
    return (row < M && col < M) ? Jp[row * M + col] : 0.f;
}

// FLIP: the scan uses the other orientation of every stored matrix than the direction's default
// (forward: J_t^T instead of J_t; reverse: J_{t+1} instead of J_{t+1}^T), so one kernel serves all
// four (direction, transpose) combinations of the bare scan.
template <int MP, bool REV, bool FLIP>
__global__ __launch_bounds__(64) void k_chunk_product_dense(const float *__restrict__ J, const float *__restrict__ rhs,
                                                            float rhs_sign, float *__restrict__ Pout,
                                                            float *__restrict__ vout, const int *__restrict__ active,
                                                            int B, int T, int M, int C, int ncs) {
    using G = DGeo<MP>;
    constexpr int NCH = G::NCH, NI = G::NI, NS = G::NS;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * NCH;
    int pb[NCH], plo[NCH], plen[NCH], us0[NCH], us1[NCH];
    int maxlen = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const int id = chain0 + n;
        bool ok = id < nchains;
        const int b = ok ? id / ncs : 0, cc = ok ? id % ncs : 0;
        ok = ok && (!active || active[b]);
        const int s0 = cc * C, s1 = min(s0 + C, T);
        const int lo = REV ? s0 + 1 : s0;
        const int hi = REV ? min(s1 + 1, T) : s1;
        pb[n] = b;
        plo[n] = lo;
        plen[n] = ok ? max(hi - lo, 0) : 0;
        us0[n] = s0;
        us1[n] = ok ? s1 : s0;
        maxlen = max(maxlen, max(plen[n], us1[n] - us0[n]));
    }
    v4f acc[NI][4];
#pragma unroll
    for (int Jt = 0; Jt < 4; ++Jt) {
        const int n = (16 * Jt) / MP;
        const int col = 16 * Jt + c - n * MP;
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[I][Jt][r] = (16 * I + 4 * g + r == col) ? 1.f : 0.f;
    }
    const int un = lane / MP, ui = lane % MP;
    int ub = 0, ulo = 0, uhi = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n)
        if (n == un) { ub = pb[n]; ulo = us0[n]; uhi = us1[n]; }
    float u = 0.f;

    for (int t = 0; t < maxlen; ++t) {
#pragma unroll
        for (int Jt = 0; Jt < 4; ++Jt) {
            const int n = (16 * Jt) / MP;
            if (t < plen[n]) {
                const float *Jp = J + ((size_t)pb[n] * T + plo[n] + t) * M * M;
                float Aop[NI][NS];
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            Aop[I][4 * j + q] = FLIP ? jload(Jp, M, 16 * j + 4 * g + q, 16 * I + c)
                                                     : jload(Jp, M, 16 * I + c, 16 * j + 4 * g + q);
                float Bop[NS];
#pragma unroll
                for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) Bop[4 * j + q] = acc[j][Jt][q];
#pragma unroll
                for (int I = 0; I < NI; ++I) {
                    v4f a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < NS; ++s) a = mfma16x16x4(Aop[I][s], Bop[s], a);
                    acc[I][Jt] = a;
                }
            }
        }
        // local solution of the chunk (lane = chain un, row ui)
        const bool run = ulo + t < uhi;
        if (!REV) {
            const int s = ulo + t;
            lds[lane] = u;
            lds_barrier();
            float y = 0.f;
            if (run && ui < M) {
                // row ui of J_s, or column ui when flipped
                const float *Jr = FLIP ? J + ((size_t)ub * T + s) * M * M + ui : J + (((size_t)ub * T + s) * M + ui) * M;
                const size_t stride = FLIP ? (size_t)M : 1;
                const float *l = lds + un * MP;
                for (int k = 0; k < M; ++k) y = fmaf(Jr[k * stride], l[k], y);
            }
            lds_barrier();
            if (run && ui < M) u = fmaf(rhs_sign, rhs[((size_t)ub * T + s) * M + ui], y);
        } else {
            const int k = uhi - 1 - t;        // y_k = J_{k+1}^T y_{k+1} + b_k
            lds[lane] = u;
            lds_barrier();
            float y = 0.f;
            if (run && ui < M && t > 0) {
                // column ui of J_{k+1}, or row ui when flipped
                const float *Jc = FLIP ? J + (((size_t)ub * T + k + 1) * M + ui) * M : J + ((size_t)ub * T + k + 1) * M * M + ui;
                const size_t stride = FLIP ? 1 : (size_t)M;
                const float *l = lds + un * MP;
                for (int r = 0; r < M; ++r) y = fmaf(Jc[r * stride], l[r], y);
            }
            lds_barrier();
            if (run && ui < M) u = fmaf(rhs_sign, rhs[((size_t)ub * T + k) * M + ui], y);
        }
    }
#pragma unroll
    for (int Jt = 0; Jt < 4; ++Jt) {
        const int n = (16 * Jt) / MP;
        const int id = chain0 + n;
        if (id < nchains && (plen[n] > 0 || us1[n] > us0[n])) {
            const int col = 16 * Jt + c - n * MP;
            float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) P[(16 * I + 4 * g + r) * MP + col] = acc[I][Jt][r];
        }
    }
    {
        const int id = chain0 + un;
        if (id < nchains) vout[(size_t)id * MP + ui] = u;
    }
}

// Forward chunk product with the chunk-local solution on the matrix cores as well: per chain
// the B operand is [P | u] (P's MP/16 column tiles plus one tile whose column 0 is u and whose
// other columns stay 0), so one set of A fragments J~_t advances both
//   P <- J~_t P,   u <- J~_t u + rhs_sign * rhs_t,
// and neither LDS nor barriers are needed.  The A fragments are read one step ahead; with the
// k-permutation kappa(4j+q, g) = 16j + 4g + q the four values a lane needs for k-steps 4j..4j+3
// are one 16-byte vector of row 16I + c.
template <int MP>
__global__ __launch_bounds__(64) void k_chunk_product_dense_fwd(const float *__restrict__ J,
                                                                const float *__restrict__ rhs, float rhs_sign,
                                                                float *__restrict__ Pout, float *__restrict__ vout,
                                                                const int *__restrict__ active, int B, int T, int M,
                                                                int C, int ncs) {
    using G = DGeo<MP>;
    constexpr int NCH = G::NCH, NI = G::NI, NS = G::NS, PT = MP / 16;
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * NCH;
    int pb[NCH], plo[NCH], plen[NCH];
    int maxlen = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const int id = chain0 + n;
        bool ok = id < nchains;
        const int b = ok ? id / ncs : 0, cc = ok ? id % ncs : 0;
        ok = ok && (!active || active[b]);
        const int s0 = cc * C, s1 = min(s0 + C, T);
        pb[n] = b;
        plo[n] = s0;
        plen[n] = ok ? max(s1 - s0, 0) : 0;
        maxlen = max(maxlen, plen[n]);
    }
    const bool vec = (M == MP);   // full 16-byte rows, no padding
    v4f acc[NCH][PT + 1][NI];
#pragma unroll
    for (int n = 0; n < NCH; ++n)
#pragma unroll
        for (int tt = 0; tt <= PT; ++tt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc[n][tt][I][r] = (tt < PT && 16 * I + 4 * g + r == 16 * tt + c) ? 1.f : 0.f;
    float an[NCH][NI][NS];   // A fragments of the next step
    float rn[NCH][NI][4];    // right-hand side of the next step (lanes of column 0)
    auto fetch = [&](int t) {
#pragma unroll
        for (int n = 0; n < NCH; ++n) {
            const bool run = t < plen[n];
            const size_t step = (size_t)pb[n] * T + plo[n] + t;
            const float *Jp = J + step * M * M;
#pragma unroll
            for (int I = 0; I < NI; ++I) {
#pragma unroll
                for (int j = 0; j < NS / 4; ++j) {
                    if (vec) {
                        const float4 v4 = run ? *reinterpret_cast<const float4 *>(Jp + (16 * I + c) * M + 16 * j + 4 * g)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
                        an[n][I][4 * j] = v4.x;
                        an[n][I][4 * j + 1] = v4.y;
                        an[n][I][4 * j + 2] = v4.z;
                        an[n][I][4 * j + 3] = v4.w;
                    } else {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            an[n][I][4 * j + q] = run ? jload(Jp, M, 16 * I + c, 16 * j + 4 * g + q) : 0.f;
                    }
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = 16 * I + 4 * g + r;
                    rn[n][I][r] = (run && c == 0 && row < M) ? rhs[step * M + row] : 0.f;
                }
            }
        }
    };
    fetch(0);
    for (int t = 0; t < maxlen; ++t) {
        float ac[NCH][NI][NS], rc[NCH][NI][4];
#pragma unroll
        for (int n = 0; n < NCH; ++n)
#pragma unroll
            for (int I = 0; I < NI; ++I) {
#pragma unroll
                for (int s = 0; s < NS; ++s) ac[n][I][s] = an[n][I][s];
#pragma unroll
                for (int r = 0; r < 4; ++r) rc[n][I][r] = rn[n][I][r];
            }
        fetch(t + 1);
#pragma unroll
        for (int n = 0; n < NCH; ++n) {
            if (t < plen[n]) {
#pragma unroll
                for (int tt = 0; tt <= PT; ++tt) {
                    float Bop[NS];
#pragma unroll
                    for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q) Bop[4 * j + q] = acc[n][tt][j][q];
#pragma unroll
                    for (int I = 0; I < NI; ++I) {
                        v4f a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int s = 0; s < NS; ++s) a = mfma16x16x4(ac[n][I][s], Bop[s], a);
                        acc[n][tt][I] = a;
                    }
                }
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[n][PT][I][r] = fmaf(rhs_sign, rc[n][I][r], acc[n][PT][I][r]);
            }
        }
    }
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const int id = chain0 + n;
        if (id >= nchains) continue;
        if (plen[n] > 0) {
            float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
            for (int tt = 0; tt < PT; ++tt)
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r = 0; r < 4; ++r) P[(16 * I + 4 * g + r) * MP + 16 * tt + c] = acc[n][tt][I][r];
        }
        if (c == 0) {
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) vout[(size_t)id * MP + 16 * I + 4 * g + r] = acc[n][PT][I][r];
        }
    }
}

// MODE 0: forward Newton fix-up (next iterate = current + Delta, in place when the two buffers
//         coincide; per-chain max |Delta| and max |z|)
// MODE 1: forward bare scan (y written)
// MODE 2: reverse (y_k = J_{k+1}^T y_{k+1} + b_k written)
// FLIP (modes 1, 2): the other orientation of the stored matrices, as in k_chunk_product_dense
template <int MP, int MODE, bool FLIP>
__global__ __launch_bounds__(64) void k_fixup_dense(const float *__restrict__ J, const float *__restrict__ rhs,
                                                    float rhs_sign, const float *__restrict__ carry_in,
                                                    float *zbuf, float *outbuf, const int *__restrict__ zsel,
                                                    uint32_t *__restrict__ chain_bits,
                                                    const int *__restrict__ active, int B, int T, int M, int C,
                                                    int ncs) {
    using G = DGeo<MP>;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * G::NCH + n;
    const bool ok0 = id < B * ncs;
    const int b = ok0 ? id / ncs : 0, cc = ok0 ? id % ncs : 0;
    const bool ok = ok0 && (!active || active[b]);
    const int s0 = cc * C, s1 = ok ? min(s0 + C, T) : s0;
    // MODE 0: iterate buffers (zbuf, outbuf) selected per sequence; MODE 1, 2: y = outbuf
    const float *zin = MODE == 0 ? cur_iter(zbuf, outbuf, zsel, b) : nullptr;
    float *out = MODE == 0 ? next_iter(zbuf, outbuf, zsel, b) : outbuf;
    float y = (ok && i < M) ? carry_in[(size_t)id * MP + i] : 0.f;
    uint32_t emax = 0u, zmax = 0u;
    const int maxlen = __builtin_amdgcn_readfirstlane(C);
    // the row (column, reverse) of J~ a step uses, its right-hand side and the iterate are
    // loaded one step ahead
    auto fetch = [&](int t, float *jv, float &bv, float &zv) {
        const int k = MODE == 2 ? s1 - 1 - t : s0 + t;
        const bool run = (MODE == 2 ? k >= s0 : k < s1) && i < M;
        const size_t e = ((size_t)b * T + k) * M + i;
        if ((MODE != 2) == FLIP) {
            // column i of J_k (forward, flipped) or of J_{k+1} (reverse)
            const int kj = MODE == 2 ? k + 1 : k;
            const bool has = run && kj < T;
            const float *Jc = J + ((size_t)b * T + kj) * M * M + i;
#pragma unroll
            for (int q = 0; q < MP; ++q) jv[q] = (has && q < M) ? Jc[(size_t)q * M] : 0.f;
        } else if (MODE != 2) {
            const float *Jr = J + (((size_t)b * T + k) * M + i) * M;
            if ((M & 3) == 0) {   // 16-byte aligned rows: vector loads
                const float4 *J4 = reinterpret_cast<const float4 *>(Jr);
#pragma unroll
                for (int q = 0; q < MP / 4; ++q) {
                    const float4 v4 = (run && 4 * q < M) ? J4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
                    jv[4 * q] = v4.x;
                    jv[4 * q + 1] = v4.y;
                    jv[4 * q + 2] = v4.z;
                    jv[4 * q + 3] = v4.w;
                }
            } else {
#pragma unroll
                for (int q = 0; q < MP; ++q) jv[q] = (run && q < M) ? Jr[q] : 0.f;
            }
        } else {
            // row i of J_{k+1} (reverse, flipped)
            const bool has = run && k + 1 < T;
            const float *Jr = J + (((size_t)b * T + k + 1) * M + i) * M;
#pragma unroll
            for (int q = 0; q < MP; ++q) jv[q] = (has && q < M) ? Jr[q] : 0.f;
        }
        bv = run ? rhs[e] : 0.f;
        zv = (MODE == 0 && run) ? zin[e] : 0.f;
    };
    float jn[MP], bn, zn;
    fetch(0, jn, bn, zn);
    for (int t = 0; t < maxlen; ++t) {
        const int k = MODE == 2 ? s1 - 1 - t : s0 + t;
        const bool run = (MODE == 2 ? k >= s0 : k < s1) && i < M;
        float jc[MP];
#pragma unroll
        for (int q = 0; q < MP; ++q) jc[q] = jn[q];
        const float bc = bn, zc = zn;
        fetch(t + 1, jn, bn, zn);
        lds[lane] = y;
        lds_barrier();
        float acc = 0.f;
        {
            const float *l = lds + n * MP;
#pragma unroll
            for (int q = 0; q < MP; ++q) acc = fmaf(jc[q], l[q], acc);
        }
        lds_barrier();
        if (run) {
            const size_t e = ((size_t)b * T + k) * M + i;
            y = fmaf(rhs_sign, bc, acc);
            if (MODE == 0) {
                const float zo = zc;
                out[e] = zo + y;
                const uint32_t ab = abs_bits(y), zb = abs_bits(zo);
                emax = emax > ab ? emax : ab;
                zmax = zmax > zb ? zmax : zb;
            } else {
                out[e] = y;
            }
        }
    }
    if (MODE == 0) {
#pragma unroll
        for (int off = MP / 2; off > 0; off >>= 1) {
            const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
            const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
            emax = emax > o ? emax : o;
            zmax = zmax > oz ? zmax : oz;
        }
        if (ok && i == 0) {   // per-chain maxima, reduced per sequence by k_seq_max
            chain_bits[id] = emax;
            chain_bits[(size_t)B * ncs + id] = zmax;
        }
    }
}

int launch_chunk_product_dense(bool rev, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                               float *P, float *v, const int *active, int C, int ncs, hipStream_t st, bool flip) {
    const int MP = padded_dim(M);
    if (MP == 128) return launch_chunk_product_big(rev, flip, B, T, M, J, rhs, rhs_sign, P, v, active, C, ncs, st);
    const int nch = B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt("k_chunk_product_dense", st);
#define CPD(MPV, R, FL)                                                                                          \
    hipLaunchKernelGGL((k_chunk_product_dense<MPV, R, FL>), dim3(grid), dim3(64), 0, st, J, rhs, rhs_sign, P, v, active, \
                       B, T, M, C, ncs)
#define CPF(MPV)                                                                                           \
    hipLaunchKernelGGL((k_chunk_product_dense_fwd<MPV>), dim3(grid), dim3(64), 0, st, J, rhs, rhs_sign, P, v, \
                       active, B, T, M, C, ncs)
    if (!rev && !flip) {
        if (MP == 16) CPF(16); else if (MP == 32) CPF(32); else CPF(64);
    } else if (!rev) {
        if (MP == 16) CPD(16, false, true); else if (MP == 32) CPD(32, false, true); else CPD(64, false, true);
    } else if (!flip) {
        if (MP == 16) CPD(16, true, false); else if (MP == 32) CPD(32, true, false); else CPD(64, true, false);
    } else {
        if (MP == 16) CPD(16, true, true); else if (MP == 32) CPD(32, true, true); else CPD(64, true, true);
    }
#undef CPF
#undef CPD
    DEER_LAUNCH_CHECK("k_chunk_product_dense");
    return DEER_OK;
}

int launch_fixup_dense(int mode, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                       const float *carry_in, float *z, float *out, const int *zsel, uint32_t *chain_bits,
                       const int *active, int C, int ncs, hipStream_t st, bool flip) {
    const int MP = padded_dim(M);
    if (MP == 128)
        return launch_fixup_big(mode, flip, B, T, M, J, rhs, rhs_sign, carry_in, z, out, zsel, chain_bits, active, C,
                                ncs, st);
    const int nch = B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt(mode == 2 ? "k_fixup_dense_rev" : "k_fixup_dense_fwd", st);
#define FXD(MPV, MO, FL)                                                                                          \
    hipLaunchKernelGGL((k_fixup_dense<MPV, MO, FL>), dim3(grid), dim3(64), 0, st, J, rhs, rhs_sign, carry_in, z, out, \
                       zsel, chain_bits, active, B, T, M, C, ncs)
#define FXD3(MO, FL) \
    if (MP == 16) FXD(16, MO, FL); else if (MP == 32) FXD(32, MO, FL); else FXD(64, MO, FL);
    if (mode == 0) { FXD3(0, false) }
    else if (mode == 1) { if (flip) { FXD3(1, true) } else { FXD3(1, false) } }
    else { if (flip) { FXD3(2, true) } else { FXD3(2, false) } }
#undef FXD3
#undef FXD
    DEER_LAUNCH_CHECK("k_fixup_dense");
    return DEER_OK;
}

}  // namespace deer
