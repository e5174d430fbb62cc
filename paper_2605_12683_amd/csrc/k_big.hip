// Latent dimensions 65..128 (padded width 128) on the stored-Jacobian path of the shallow PLRNN:
// the same operations as the M <= 64 kernels (k_dense.hip, k_shallow.hip, the carry walk), laid
// out for a 128 x 128 chain matrix that one wave cannot hold.
//
//   k_chunk_product_big   one 4-wave workgroup per chain: wave w holds columns 32w..32w+31 of the
//                         chunk product P <- E_t P in matrix-core accumulators (the previous step's
//                         accumulators are the B operand, the step's Jacobian rows the A operand,
//                         read as 16-byte vectors); the chunk-local solution u <- E_t u + rhs on
//                         the vector units through LDS
//   k_carry_big           one 256-thread block per walk: carries across the chunks, one level,
//                         or two with k_carry_group_big (group maps on the matrix cores)
//   k_fixup_big           one 128-thread block per chain: each chunk re-run from its carry
//   k_resjac_big          residual, masks (the fixed-order float32 decision) and F, one row per
//                         wave, W1 and W2 in LDS
//   k_jacform_big         J~ = diag(A p) + W1 diag(m) (W2 P) on the matrix cores, 4 waves per
//                         row, two column tiles each
//   k_grads_big           per-block partial sums of the shallow gradients (layout of
//                         k_grads_shplrnn), summed by k_reduce_rows
// E_t is J_t, or J_t^T when flipped (the bare scan's other orientation), as in k_dense.hip.
#include "common.h"
#include "launch.h"

namespace deer {

constexpr int BG = 128;   // padded width
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// element (row, col) of E_t (J_t row-major per step, zero outside M x M)
template <bool FLIP>
__device__ __forceinline__ float eload(const float *__restrict__ Jp, int M, int row, int col) {
    if (row >= M || col >= M) return 0.f;
    return FLIP ? Jp[(size_t)col * M + row] : Jp[(size_t)row * M + col];
}

// REV: the product covers steps [s0 + 1, min(s1 + 1, T)) (the reverse chunk map is its
// transpose) and the local solution of u_k = E_{k+1}^T u_{k+1} + rhs_k (zero past the chunk) is
// taken as the sum u_{s0} = sum_k (E_k ... E_{s0+1})^T rhs_k along the same sweep.
// The step's E (128 x 128, zero outside M x M) is staged in LDS by the whole workgroup, the next
// step's loads in flight while the matrix cores work on this one (double buffer), and every wave
// reads its A operands there; the forward local solution reads the same tile.
constexpr int JST = BG + 4;   // LDS row stride of the staged E (16-byte rows, conflict-free reads)

template <bool REV, bool FLIP>
__global__ __launch_bounds__(256) void k_chunk_product_big(const float *__restrict__ J, const float *__restrict__ rhs,
                                                           float rhs_sign, float *__restrict__ Pout,
                                                           float *__restrict__ vout, const int *__restrict__ active,
                                                           int B, int T, int M, int C, int ncs) {
    __shared__ __align__(16) float js[2][BG][JST];
    __shared__ __align__(16) float ub[2][BG];
    const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int id = blockIdx.x;   // chain
    const int b = id / ncs, cc = id % ncs;
    const bool ok = !active || active[b];
    const int s0 = cc * C, s1 = min(s0 + C, T);
    const int lo = REV ? s0 + 1 : s0, hi = REV ? min(s1 + 1, T) : s1;
    const int plen = ok ? max(hi - lo, 0) : 0;
    const int ulen = ok ? s1 - s0 : 0;
    // REV: the chunk's local adjoint is u_{s0} = sum_k Q_k^T rhs_k with Q_k = E_k ... E_{s0+1}
    // (Q_{s0} = I), and Q_k is the accumulated product after the step that takes E_k: the sweep
    // that forms the product forms u_{s0} too, with the staged right-hand side of that step
    const int nsteps = REV ? plen : max(plen, ulen);
    // staging: thread tid takes the 16-byte groups tid + 256 k (k < 16) of the 128 x 128 tile,
    // row (tid + 256 k) / 32, columns 4 ((tid + 256 k) % 32) .. + 3
    float4 pre[16];
    float rpre = 0.f;
    // row-major E with M % 4 == 0: 16-byte loads through a resource bounded at the matrix's end
    // (rows past M read zero) with one lane offset (columns past M: an offset outside it)
    const bool fast = !FLIP && (M & 3) == 0;
    const uint32_t vlane = ((tid & 31) * 4 + 3 < M) ? 4u * ((uint32_t)(tid >> 5) * M + (tid & 31) * 4) : kOffLane;
    auto stage_load = [&](int t) {
        const float *Jp = J + ((size_t)b * T + lo + t) * M * M;
        if (REV) rpre = (tid < M && lo + t < s1) ? rhs[((size_t)b * T + lo + t) * M + tid] : 0.f;
        if (fast) {
            const auto rs = bounded_rsrc(Jp, (uint32_t)M * M * 4u);
#pragma unroll
            for (int k = 0; k < 16; ++k)
                pre[k] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)vlane, k * 32 * M, 0));
            return;
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int e4 = tid + 256 * k, row = e4 >> 5, c4 = (e4 & 31) * 4;
            pre[k] = make_float4(eload<FLIP>(Jp, M, row, c4), eload<FLIP>(Jp, M, row, c4 + 1),
                                 eload<FLIP>(Jp, M, row, c4 + 2), eload<FLIP>(Jp, M, row, c4 + 3));
        }
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int e4 = tid + 256 * k;
            *reinterpret_cast<float4 *>(&js[buf][e4 >> 5][(e4 & 31) * 4]) = pre[k];
        }
        if (REV && tid < BG) ub[buf][tid] = rpre;
    };
    // accumulators: acc[I][Jt][r] = P[16 I + 4 g + r][32 wv + 16 Jt + c]
    v4f acc[8][2];
#pragma unroll
    for (int I = 0; I < 8; ++I)
#pragma unroll
        for (int Jt = 0; Jt < 2; ++Jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[I][Jt][r] = (16 * I + 4 * g + r == 32 * wv + 16 * Jt + c) ? 1.f : 0.f;
    // local solution: thread pair (row i = tid / 2, half hh) sums half of the row
    const int ui = tid >> 1, hh = tid & 1;
    if (tid < BG) ub[0][tid] = 0.f;
    float vsum[2] = {0.f, 0.f};   // REV: sum over the steps of (Q_k^T rhs_k)[32 wv + 16 Jt + c]
    if (plen > 0) {
        stage_load(0);
        stage_store(0);
    }
    __syncthreads();
    int cur = 0;
    for (int t = 0; t < nsteps; ++t) {
        const bool more = t + 1 < plen;
        if (more) stage_load(t + 1);   // in flight during this step
        if (t < plen) {
            v4f old[8][2];
#pragma unroll
            for (int I = 0; I < 8; ++I)
#pragma unroll
                for (int Jt = 0; Jt < 2; ++Jt) {
                    old[I][Jt] = acc[I][Jt];
                    acc[I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
            for (int I = 0; I < 8; ++I) {
                float4 a[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) a[j] = *reinterpret_cast<const float4 *>(&js[cur][16 * I + c][16 * j + 4 * g]);
#pragma unroll
                for (int Jt = 0; Jt < 2; ++Jt) {
                    v4f s = acc[I][Jt];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        s = mfma16x16x4(a[j].x, old[j][Jt][0], s);
                        s = mfma16x16x4(a[j].y, old[j][Jt][1], s);
                        s = mfma16x16x4(a[j].z, old[j][Jt][2], s);
                        s = mfma16x16x4(a[j].w, old[j][Jt][3], s);
                    }
                    acc[I][Jt] = s;
                }
            }
            if (REV && lo + t < s1) {
                // rows 16 I + 4 g + r of column 32 wv + 16 Jt + c, then the four row groups g
#pragma unroll
                for (int Jt = 0; Jt < 2; ++Jt) {
                    float part = 0.f;
#pragma unroll
                    for (int I = 0; I < 8; ++I) {
                        const float4 rv = *reinterpret_cast<const float4 *>(&ub[cur][16 * I + 4 * g]);
                        part = fmaf(acc[I][Jt][0], rv.x, part);
                        part = fmaf(acc[I][Jt][1], rv.y, part);
                        part = fmaf(acc[I][Jt][2], rv.z, part);
                        part = fmaf(acc[I][Jt][3], rv.w, part);
                    }
                    part += __shfl_xor(part, 16, 64);
                    part += __shfl_xor(part, 32, 64);
                    vsum[Jt] += part;
                }
            }
        }
        if (!REV && t < ulen) {
            // u_s = E_s u_{s-1} + sign rhs_s, s = s0 + t (E_s is the staged tile, zero outside M x M
            // as u is): half hh of row ui, q in [64 hh, 64 hh + 64) four at a time, walked from 32
            // entries in for hh = 1 so that the two halves of a lane pair fall on other banks
            const int k = s0 + t;
            float p0 = 0.f, p1 = 0.f;
#pragma unroll 4
            for (int u = 0; u < 64; u += 4) {
                const int q = 64 * hh + ((u + 32 * hh) & 63);
                const float4 e = *reinterpret_cast<const float4 *>(&js[cur][ui][q]);
                const float4 y = *reinterpret_cast<const float4 *>(&ub[cur][q]);
                p0 = fmaf(e.x, y.x, p0);
                p1 = fmaf(e.y, y.y, p1);
                p0 = fmaf(e.z, y.z, p0);
                p1 = fmaf(e.w, y.w, p1);
            }
            float part = p0 + p1;
            part += __shfl_xor(part, 1, 64);
            if (hh == 0 && ui < BG)
                ub[cur ^ 1][ui] = ui < M ? fmaf(rhs_sign, rhs[((size_t)b * T + k) * M + ui], part) : 0.f;
        }
        if (more) stage_store(cur ^ 1);   // that buffer's reads ended at the previous barrier
        __syncthreads();
        cur ^= 1;
    }
    if (!ok) return;
    float *P = Pout + (size_t)id * BG * BG;
#pragma unroll
    for (int I = 0; I < 8; ++I)
#pragma unroll
        for (int Jt = 0; Jt < 2; ++Jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) P[(16 * I + 4 * g + r) * BG + 32 * wv + 16 * Jt + c] = acc[I][Jt][r];
    if (REV) {
        if (g == 0) {
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) {
                const int col = 32 * wv + 16 * Jt + c;
                const float r0 = (col < M && s0 < s1) ? rhs[((size_t)b * T + s0) * M + col] : 0.f;
                vout[(size_t)id * BG + col] = col < M ? rhs_sign * (r0 + vsum[Jt]) : 0.f;
            }
        }
    } else if (tid < BG) {
        vout[(size_t)id * BG + tid] = ub[cur][tid];
    }
}

// carries across the chunks of each sequence, in processing order k (REV: chunk c = ncs - 1 - k):
// carry_in[c] = the state entering chunk c;  next = A_k carry + v_c with A_k = P_c (P_c^T in REV).
// Long chunk sequences use two levels: groups of G consecutive k composed into one map (Q_j, u_j)
// on the matrix cores (k_carry_group_big, all groups in parallel), a walk over the group maps, and
// every group re-walked from its carry.  Serial depth G + ncs / G + G instead of ncs.
constexpr int FST = BG + 1;   // LDS row stride of a tile read along rows and along columns

// one walk of G consecutive k per 256-thread block (G = ncs: a whole sequence), from zero or from
// the walk's start vector.  Lane l of wave w forms half hh = l / 32 of row i = 32 w + l % 32 of
// A_k y; each step's P_c is staged in LDS with coalesced loads, the next one's in flight.
template <bool REV>
__global__ __launch_bounds__(256) void k_carry_big(const float *__restrict__ P, const float *__restrict__ v,
                                                   float *__restrict__ carry_in, const int *__restrict__ active,
                                                   int ncs, int G, const float *__restrict__ start) {
    __shared__ float js[2][BG][FST];
    __shared__ float ys[2][BG];
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hh = lane >> 5, i = 32 * w + (lane & 31);
    if (active && !active[b]) return;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    auto chunk = [&](int k) { return (size_t)b * ncs + (REV ? ncs - 1 - k : k); };
    // staging: thread tid takes the 16-byte groups tid + 256 q (q < 16) of the 128 x 128 map,
    // row (tid + 256 q) / 32, columns 4 (tid % 32) .. + 3
    float4 pre[16];
    float vpre = 0.f;
    auto stage_load = [&](int k) {
        const size_t id = chunk(k);
        const float4 *P4 = reinterpret_cast<const float4 *>(P + id * BG * BG);
#pragma unroll
        for (int q = 0; q < 16; ++q) pre[q] = P4[tid + 256 * q];
        vpre = v[id * BG + i];
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int e4 = tid + 256 * q, row = e4 >> 5, c4 = (e4 & 31) * 4;
            js[buf][row][c4] = pre[q].x;
            js[buf][row][c4 + 1] = pre[q].y;
            js[buf][row][c4 + 2] = pre[q].z;
            js[buf][row][c4 + 3] = pre[q].w;
        }
    };
    if (tid < BG) ys[0][tid] = start ? start[((size_t)b * ngroups + j) * BG + tid] : 0.f;
    stage_load(k0);
    stage_store(0);
    float vc = vpre;
    __syncthreads();
    int cur = 0;
    const int q0 = 64 * hh;
    for (int k = k0; k < k1; ++k) {
        const bool more = k + 1 < k1;
        if (more) stage_load(k + 1);   // in flight during this step
        if (hh == 0) carry_in[chunk(k) * BG + i] = ys[cur][i];
        // half hh of the sum over q in [64 hh, 64 hh + 64), walked from 32 hh on: with the row
        // stride of 129 the 64 lanes of a read fall on distinct banks, along rows and columns
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll 4
        for (int u = 0; u < 64; u += 4) {
            const int q = q0 + ((u + 32 * hh) & 63);
            const float e0 = REV ? js[cur][q][i] : js[cur][i][q];
            const float e1 = REV ? js[cur][q + 1][i] : js[cur][i][q + 1];
            const float e2 = REV ? js[cur][q + 2][i] : js[cur][i][q + 2];
            const float e3 = REV ? js[cur][q + 3][i] : js[cur][i][q + 3];
            a0 = fmaf(e0, ys[cur][q], a0);
            a1 = fmaf(e1, ys[cur][q + 1], a1);
            a2 = fmaf(e2, ys[cur][q + 2], a2);
            a3 = fmaf(e3, ys[cur][q + 3], a3);
        }
        float part = (a0 + a1) + (a2 + a3);
        part += __shfl_xor(part, 32, 64);
        if (hh == 0) ys[cur ^ 1][i] = part + vc;
        if (more) {
            stage_store(cur ^ 1);   // that buffer's reads ended at the previous barrier
            vc = vpre;
        }
        __syncthreads();
        cur ^= 1;
    }
}

// group maps in processing order: Q_j = A_{k1-1} ... A_{k0} and u_j = the group's walk from zero.
// Q accumulates on the matrix cores as the chunk product above does (A_k staged in LDS, transposed
// there in REV, the next one's loads in flight; Q in the k-permuted accumulator layout that is the
// next step's B operand); u by thread pairs over the staged rows.
template <bool REV>
__global__ __launch_bounds__(256) void k_carry_group_big(const float *__restrict__ P, const float *__restrict__ v,
                                                         float *__restrict__ gq, float *__restrict__ gu,
                                                         const int *__restrict__ active, int ncs, int G) {
    __shared__ __align__(16) float js[2][BG][JST];
    __shared__ __align__(16) float ub[2][BG];
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups;
    const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    if (active && !active[b]) return;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    auto chunk = [&](int k) { return (size_t)b * ncs + (REV ? ncs - 1 - k : k); };
    const int ui = tid >> 1, hh = tid & 1;
    float4 pre[16];
    float vpre = 0.f;
    auto stage_load = [&](int k) {
        const size_t id = chunk(k);
        const float4 *P4 = reinterpret_cast<const float4 *>(P + id * BG * BG);
#pragma unroll
        for (int q = 0; q < 16; ++q) pre[q] = P4[tid + 256 * q];
        if (hh == 0) vpre = v[id * BG + ui];
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int e4 = tid + 256 * q, row = e4 >> 5, c4 = (e4 & 31) * 4;
            if (REV) {
                js[buf][c4][row] = pre[q].x;
                js[buf][c4 + 1][row] = pre[q].y;
                js[buf][c4 + 2][row] = pre[q].z;
                js[buf][c4 + 3][row] = pre[q].w;
            } else {
                *reinterpret_cast<float4 *>(&js[buf][row][c4]) = pre[q];
            }
        }
    };
    // accumulators: acc[I][Jt][r] = Q[16 I + 4 g + r][32 wv + 16 Jt + c]
    v4f acc[8][2];
#pragma unroll
    for (int I = 0; I < 8; ++I)
#pragma unroll
        for (int Jt = 0; Jt < 2; ++Jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[I][Jt][r] = (16 * I + 4 * g + r == 32 * wv + 16 * Jt + c) ? 1.f : 0.f;
    if (tid < BG) ub[0][tid] = 0.f;
    stage_load(k0);
    stage_store(0);
    float vc = vpre;
    __syncthreads();
    int cur = 0;
    for (int k = k0; k < k1; ++k) {
        const bool more = k + 1 < k1;
        if (more) stage_load(k + 1);   // in flight during this step
        v4f old[8][2];
#pragma unroll
        for (int I = 0; I < 8; ++I)
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) {
                old[I][Jt] = acc[I][Jt];
                acc[I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
        for (int I = 0; I < 8; ++I) {
            float4 a[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) a[jj] = *reinterpret_cast<const float4 *>(&js[cur][16 * I + c][16 * jj + 4 * g]);
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) {
                v4f s = acc[I][Jt];
#pragma unroll
                for (int jj = 0; jj < 8; ++jj) {
                    s = mfma16x16x4(a[jj].x, old[jj][Jt][0], s);
                    s = mfma16x16x4(a[jj].y, old[jj][Jt][1], s);
                    s = mfma16x16x4(a[jj].z, old[jj][Jt][2], s);
                    s = mfma16x16x4(a[jj].w, old[jj][Jt][3], s);
                }
                acc[I][Jt] = s;
            }
        }
        // u <- A_k u + v_c: thread pair (row ui, half hh) sums every other entry of the row
        float part = 0.f;
        for (int q = hh; q < BG; q += 2) part = fmaf(js[cur][ui][q], ub[cur][q], part);
        part += __shfl_xor(part, 1, 64);
        if (hh == 0) ub[cur ^ 1][ui] = part + vc;
        if (more) {
            stage_store(cur ^ 1);   // that buffer's reads ended at the previous barrier
            vc = vpre;
        }
        __syncthreads();
        cur ^= 1;
    }
    float *q = gq + ((size_t)b * ngroups + j) * BG * BG;
#pragma unroll
    for (int I = 0; I < 8; ++I)
#pragma unroll
        for (int Jt = 0; Jt < 2; ++Jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) q[(16 * I + 4 * g + r) * BG + 32 * wv + 16 * Jt + c] = acc[I][Jt][r];
    if (tid < BG) gu[((size_t)b * ngroups + j) * BG + tid] = ub[cur][tid];
}

// MODE 0: Newton fix-up (next iterate = current + Delta, per-chain max |Delta| and max |z|);
// MODE 1: forward bare scan; MODE 2: reverse (y_k = E_{k+1}^T y_{k+1} + b_k).  256 threads: lane
// l of wave w forms half hh = l / 32 of row i = 32 w + l % 32 of E y (MODE 2: of E^T y), the two
// halves added across the wave.  Each step's E is staged in LDS by the block with coalesced
// loads, the next step's loads (and its right-hand side and iterate) in flight during this step.
// With a row stride of 129 floats and the second half's walk started 32 entries in, the 64 lanes
// of a read fall on distinct banks, for rows (MODE 0, 1) and for columns (MODE 2).

template <int MODE, bool FLIP>
__global__ __launch_bounds__(256) void k_fixup_big(const float *__restrict__ J, const float *__restrict__ rhs,
                                                   float rhs_sign, const float *__restrict__ carry_in, float *zbuf,
                                                   float *outbuf, const int *__restrict__ zsel,
                                                   uint32_t *__restrict__ chain_bits, const int *__restrict__ active,
                                                   int B, int T, int M, int C, int ncs) {
    __shared__ float js[2][BG][FST];
    __shared__ float ys[2][BG];
    __shared__ uint32_t red[2][4];
    const int id = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int hh = lane >> 5, i = 32 * w + (lane & 31);
    const int b = id / ncs, cc = id % ncs;
    const bool ok = !active || active[b];
    const int s0 = cc * C, s1 = ok ? min(s0 + C, T) : s0;
    const int len = s1 - s0;
    const float *zin = MODE == 0 ? cur_iter(zbuf, outbuf, zsel, b) : nullptr;
    float *out = MODE == 0 ? next_iter(zbuf, outbuf, zsel, b) : outbuf;
    const bool own = hh == 0 && i < M;   // the lane that writes row i
    // step t: k = the row of the output, kj = the matrix (MODE 2: k + 1, none past the end)
    auto k_of = [&](int t) { return MODE == 2 ? s1 - 1 - t : s0 + t; };
    // staging: thread tid takes the 16-byte groups tid + 256 q (q < 16), row (tid + 256 q) / 32
    float4 pre[16];
    float rpre = 0.f, zpre = 0.f;
    // row-major E with M % 4 == 0: 16-byte loads through a resource bounded at the matrix's end
    // (rows past M read zero) with one lane offset (columns past M: an offset outside it)
    const bool fast = !FLIP && (M & 3) == 0;
    const uint32_t vlane = ((tid & 31) * 4 + 3 < M) ? 4u * ((uint32_t)(tid >> 5) * M + (tid & 31) * 4) : kOffLane;
    auto stage_load = [&](int t) {
        const int k = k_of(t), kj = MODE == 2 ? k + 1 : k;
        const bool has = kj < T;
        const float *Jp = J + ((size_t)b * T + (has ? kj : 0)) * M * M;
        if (fast) {
            const auto rs = bounded_rsrc(Jp, has ? (uint32_t)M * M * 4u : 0u);
#pragma unroll
            for (int q = 0; q < 16; ++q)
                pre[q] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)vlane, q * 32 * M, 0));
        } else {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int e4 = tid + 256 * q, row = e4 >> 5, c4 = (e4 & 31) * 4;
                pre[q] = !has ? make_float4(0.f, 0.f, 0.f, 0.f)
                              : make_float4(eload<FLIP>(Jp, M, row, c4), eload<FLIP>(Jp, M, row, c4 + 1),
                                            eload<FLIP>(Jp, M, row, c4 + 2), eload<FLIP>(Jp, M, row, c4 + 3));
            }
        }
        if (own) {
            const size_t e = ((size_t)b * T + k) * M + i;
            rpre = rhs[e];
            if (MODE == 0) zpre = zin[e];
        }
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int e4 = tid + 256 * q, row = e4 >> 5, c4 = (e4 & 31) * 4;
            js[buf][row][c4] = pre[q].x;
            js[buf][row][c4 + 1] = pre[q].y;
            js[buf][row][c4 + 2] = pre[q].z;
            js[buf][row][c4 + 3] = pre[q].w;
        }
    };
    if (tid < BG) ys[0][tid] = (ok && tid < M) ? carry_in[(size_t)id * BG + tid] : 0.f;
    float rc = 0.f, zc = 0.f;
    if (len > 0) {
        stage_load(0);
        stage_store(0);
        rc = rpre;
        zc = zpre;
    }
    __syncthreads();
    uint32_t emax = 0u, zmax = 0u;
    int cur = 0;
    const int q0 = 64 * hh;
    for (int t = 0; t < len; ++t) {
        const int k = k_of(t);
        const bool more = t + 1 < len;
        if (more) stage_load(t + 1);   // in flight during this step
        // half hh of the sum over q in [64 hh, 64 hh + 64), walked from 32 hh on (entries past M
        // are zero in the staged tile and in ys)
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll 4
        for (int u = 0; u < 64; u += 4) {
            const int q = q0 + ((u + 32 * hh) & 63);
            const float e0 = MODE == 2 ? js[cur][q][i] : js[cur][i][q];
            const float e1 = MODE == 2 ? js[cur][q + 1][i] : js[cur][i][q + 1];
            const float e2 = MODE == 2 ? js[cur][q + 2][i] : js[cur][i][q + 2];
            const float e3 = MODE == 2 ? js[cur][q + 3][i] : js[cur][i][q + 3];
            a0 = fmaf(e0, ys[cur][q], a0);
            a1 = fmaf(e1, ys[cur][q + 1], a1);
            a2 = fmaf(e2, ys[cur][q + 2], a2);
            a3 = fmaf(e3, ys[cur][q + 3], a3);
        }
        float part = (a0 + a1) + (a2 + a3);
        part += __shfl_xor(part, 32, 64);
        float y = 0.f;
        if (own) {
            const size_t e = ((size_t)b * T + k) * M + i;
            y = fmaf(rhs_sign, rc, part);
            if (MODE == 0) {
                out[e] = zc + y;
                const uint32_t ab = abs_bits(y), zb = abs_bits(zc);
                emax = emax > ab ? emax : ab;
                zmax = zmax > zb ? zmax : zb;
            } else {
                out[e] = y;
            }
        }
        if (hh == 0) ys[cur ^ 1][i] = y;
        if (more) {
            stage_store(cur ^ 1);   // that buffer's reads ended at the previous barrier
            rc = rpre;
            zc = zpre;
        }
        __syncthreads();
        cur ^= 1;
    }
    if (MODE == 0) {
        emax = wave_max_u32(emax);
        zmax = wave_max_u32(zmax);
        if (lane == 0) {
            red[0][w] = emax;
            red[1][w] = zmax;
        }
        __syncthreads();
        if (tid == 0 && ok) {
            uint32_t e = red[0][0], z = red[1][0];
            for (int v = 1; v < 4; ++v) {
                e = e > red[0][v] ? e : red[0][v];
                z = z > red[1][v] ? z : red[1][v];
            }
            chain_bits[id] = e;
            chain_bits[(size_t)B * ncs + id] = z;
        }
    }
}

// ---- shallow PLRNN at M <= 128 -------------------------------------------------------------

// forced input of step s for latent i, the float32 decision of the other kernels
__device__ __forceinline__ float big_forced(const ShArgs &a, const float *z, int b, int s, int i) {
    if (s == 0) return a.z0 ? a.z0[(size_t)b * a.M + i] : (i < a.N ? a.x[(size_t)b * (a.T + 1) * a.N + i] : 0.f);
    if (a.zt) return a.zt[((size_t)b * a.T + s) * a.M + i];
    const float zp = z[((size_t)b * a.T + s - 1) * a.M + i];
    if (i >= a.N) return zp;
    const float xs = a.x[((size_t)b * (a.T + 1) + s) * a.N + i];
    if (s <= a.tw) return xs;   // latent warm-up: alpha_s = 1
    const float p = __fsub_rn(1.0f, a.alpha);
    return __fadd_rn(__fmul_rn(p, zp), __fmul_rn(a.alpha, xs));
}

// One row per wave, the four waves of a block on their own rows; LDS: W2^T [M][L] | W1^T [L][M],
// so that the lanes of a read take consecutive words.  Lane l < L forms the hidden pre-activation
// u_l left to right from h2 (a rounding after every multiply and add: the fixed-order float32
// decision), with z~_j broadcast from lane j % 64 of the wave's registers; lanes i and i + 64 form
// F_i and r_i from relu(u), broadcast the same way.
__global__ __launch_bounds__(256) void k_resjac_big(const ShArgs a, const float *zbuf, const float *zalt,
                                                    const int *__restrict__ zsel, float *__restrict__ F_out,
                                                    float *__restrict__ r_out, uint32_t *__restrict__ masks,
                                                    const int *__restrict__ active) {
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    float *w2t = smem, *w1t = w2t + (size_t)M * L;
    for (int e = tid; e < M * L; e += 256) {
        const int i = e / L, l = e % L;   // W1[i][l]; W2[l][i] at the same (i, l)
        w1t[(size_t)l * M + i] = a.W1[e];
        w2t[(size_t)i * L + l] = a.W2[(size_t)l * M + i];
    }
    const int LW = (L + 31) / 32;
    const long rows = (long)a.B * T;
    __syncthreads();
    for (long row = (long)blockIdx.x * 4 + wv; row < rows; row += (long)gridDim.x * 4) {
        const int b = (int)(row / T), s = (int)(row % T);
        if (active && !active[b]) continue;   // wave-uniform
        const float *z = cur_iter(zbuf, zalt, zsel, b);
        const int i1 = lane + 64;
        const float zt0 = lane < M ? big_forced(a, z, b, s, lane) : 0.f;
        const float zt1 = i1 < M ? big_forced(a, z, b, s, i1) : 0.f;
        float u = 0.f;
        if (lane < L) {
            u = a.h2 ? a.h2[lane] : 0.f;
            const float *wr = w2t + lane;
            const int m0 = M < 64 ? M : 64;
            for (int j = 0; j < m0; ++j)
                u = __fadd_rn(u, __fmul_rn(wr[(size_t)j * L], __int_as_float(__builtin_amdgcn_readlane(__float_as_int(zt0), j))));
            for (int j = 64; j < M; ++j)
                u = __fadd_rn(u, __fmul_rn(wr[(size_t)j * L], __int_as_float(__builtin_amdgcn_readlane(__float_as_int(zt1), j - 64))));
        }
        const float ru = (lane < L && u > 0.f) ? u : 0.f;
        const uint64_t on = __builtin_amdgcn_ballot_w64(lane < L && u > 0.f);
        if (masks && lane < LW) masks[(size_t)row * LW + lane] = (uint32_t)(on >> (32 * lane));
        float f0 = 0.f, f1 = 0.f;
        for (int l = 0; l < L; ++l) {
            const float rl = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ru), l));
            f0 = fmaf(w1t[(size_t)l * M + lane], rl, f0);
            if (i1 < M) f1 = fmaf(w1t[(size_t)l * M + i1], rl, f1);
        }
        const size_t e0 = (size_t)row * M;
        if (lane < M) {
            const float f = fmaf(a.A[lane], zt0, f0) + (a.h1 ? a.h1[lane] : 0.f);
            if (F_out) F_out[e0 + lane] = f;
            if (r_out) r_out[e0 + lane] = z[e0 + lane] - f;
        }
        if (i1 < M) {
            const float f = fmaf(a.A[i1], zt1, f1) + (a.h1 ? a.h1[i1] : 0.f);
            if (F_out) F_out[e0 + i1] = f;
            if (r_out) r_out[e0 + i1] = z[e0 + i1] - f;
        }
    }
}

// J~_s = Cd (or diag(A p)) + W1 diag(m_s) V with V = W2 diag(p) (or the given W2 P): one row at a
// time per block, the blocks walking the rows, wave wv computes the column tiles 2 wv, 2 wv + 1 of all 8 row tiles.  LDS: W1 [BG][LP],
// V^T [BG][LP], zero padded (LP = L rounded up to 16).
template <bool ROW4>
__global__ __launch_bounds__(256) void k_jacform_big(const ShArgs a, const uint32_t *__restrict__ masks,
                                                     float *__restrict__ Jout, const int *__restrict__ active,
                                                     const float *__restrict__ gamma, int LP) {
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, N = a.N;
    float *w1s = smem, *vts = smem + BG * LP;
    const int tid = threadIdx.x;
    const float p1 = __fsub_rn(1.0f, a.alpha);
    for (int e = tid; e < BG * LP; e += 256) {
        const int i = e / LP, l = e % LP;
        const bool in = i < M && l < L;
        w1s[e] = in ? a.W1[(size_t)i * L + l] : 0.f;
        vts[e] = in ? a.W2[(size_t)l * M + i] * (i < N ? p1 : 1.f) : 0.f;
    }
    __syncthreads();
    const int wv = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    const auto cd_rs = bounded_rsrc(a.Cd, a.Cd ? (uint32_t)M * M * 4u : 0u);
    // diagonal A p of rows 16 I + c (the transposed-tile stores)
    float dgI[8];
#pragma unroll
    for (int I = 0; I < 8; ++I) {
        const int i = 16 * I + c;
        dgI[I] = (ROW4 && !a.Cd && i < M) ? a.A[i] * (i < N ? p1 : 1.f) : 0.f;
    }
    const int t_lo = a.t_hi > a.t_lo ? a.t_lo : 0;
    const int len = a.t_hi > a.t_lo ? a.t_hi - a.t_lo : T;
    const long rows = (long)a.B * len;
    auto grow_of = [&](long r) {
        const long bb = r / len;
        return bb * T + t_lo + (r - bb * len);
    };
    // the next row's mask words (L <= 64: at most two) are loaded while this row is formed
    uint32_t wn0 = 0u, wn1 = 0u;
    auto fetch = [&](long r) {
        if (r >= rows) return;
        const uint32_t *mw = masks + (size_t)grow_of(r) * LW;
        wn0 = mw[0];
        wn1 = LW > 1 ? mw[1] : 0u;
    };
    fetch(blockIdx.x);
    for (long r0 = blockIdx.x; r0 < rows; r0 += gridDim.x) {
        const long bb = r0 / len;
        const long grow = grow_of(r0);
        const uint32_t wc0 = wn0, wc1 = wn1;
        fetch(r0 + gridDim.x);
        if (active && !active[bb]) continue;
        v4f acc[8][2];
#pragma unroll
        for (int I = 0; I < 8; ++I)
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) acc[I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int j = 0; j < LP / 16; ++j) {
            const int sh = 16 * (j & 1) + 4 * g;
            const uint32_t w = j < 2 ? wc0 : wc1;
            float4 bv[2];
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) {
                const float4 t4 = *reinterpret_cast<const float4 *>(vts + (32 * wv + 16 * Jt + c) * LP + 16 * j + 4 * g);
                bv[Jt] = make_float4(select_bit(w, sh, t4.x), select_bit(w, sh + 1, t4.y), select_bit(w, sh + 2, t4.z),
                                     select_bit(w, sh + 3, t4.w));
            }
#pragma unroll
            for (int I = 0; I < 8; ++I) {
                const float4 av = *reinterpret_cast<const float4 *>(w1s + (16 * I + c) * LP + 16 * j + 4 * g);
#pragma unroll
                for (int Jt = 0; Jt < 2; ++Jt) {
                    v4f t = acc[I][Jt];
                    if (ROW4) {   // the transposed tile: V^T diag(m) W1^T
                        t = mfma16x16x4(bv[Jt].x, av.x, t);
                        t = mfma16x16x4(bv[Jt].y, av.y, t);
                        t = mfma16x16x4(bv[Jt].z, av.z, t);
                        t = mfma16x16x4(bv[Jt].w, av.w, t);
                    } else {
                        t = mfma16x16x4(av.x, bv[Jt].x, t);
                        t = mfma16x16x4(av.y, bv[Jt].y, t);
                        t = mfma16x16x4(av.z, bv[Jt].z, t);
                        t = mfma16x16x4(av.w, bv[Jt].w, t);
                    }
                    acc[I][Jt] = t;
                }
            }
        }
        // stores through a resource bounded at J~_s's end: rows past M fall outside it, columns
        // past M take an offset outside it
        const auto rs = bounded_rsrc(Jout + (size_t)grow * M * M, (uint32_t)M * M * 4u);
        const float gm = gamma ? gamma[bb] : 1.f;
        if (ROW4) {
            // acc[I][Jt][r] = J~[16 I + c][32 wv + 16 Jt + 4 g + r]: one 16-byte store per tile (with
            // M % 4 == 0 the four columns are all inside the row or all past it)
#pragma unroll
            for (int Jt = 0; Jt < 2; ++Jt) {
                const int col0 = 32 * wv + 16 * Jt + 4 * g;
                const uint32_t vo = col0 < M ? 4u * (uint32_t)(c * M + col0) : kOffLane;
#pragma unroll
                for (int I = 0; I < 8; ++I) {
                    const uint32_t vr = vo + 4u * (uint32_t)M * (uint32_t)(16 * I);
                    const int dr = 16 * I + c - col0;   // the diagonal entry's column in the four
                    float4 d = make_float4(dr == 0 ? dgI[I] : 0.f, dr == 1 ? dgI[I] : 0.f, dr == 2 ? dgI[I] : 0.f,
                                           dr == 3 ? dgI[I] : 0.f);
                    if (a.Cd) d = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(cd_rs, (int)vr, 0, 0));
                    const float4 o = make_float4(gm * (acc[I][Jt][0] + d.x), gm * (acc[I][Jt][1] + d.y),
                                                 gm * (acc[I][Jt][2] + d.z), gm * (acc[I][Jt][3] + d.w));
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, o), rs, (int)vr, 0, 0);
                }
            }
            continue;
        }
#pragma unroll
        for (int Jt = 0; Jt < 2; ++Jt) {
            const int col = 32 * wv + 16 * Jt + c;
            const uint32_t vo = col < M ? 4u * (uint32_t)(4 * g * M + col) : kOffLane;
            // the diagonal entry (col, col) sits in row tile col / 16 at 4 g + r = col % 16
            const float dg = (!a.Cd && col < M) ? a.A[col] * (col < N ? p1 : 1.f) : 0.f;
#pragma unroll
            for (int I = 0; I < 8; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    // lane offset of row 16 I + 4 g + r (kOffLane plus a row offset stays outside)
                    const uint32_t vr = vo + 4u * (uint32_t)M * (uint32_t)(16 * I + r);
                    float d = (16 * I + 4 * g + r == col) ? dg : 0.f;
                    if (a.Cd) d = bload(cd_rs, vr, 0);
                    bstore_u(rs, __float_as_uint(gm * (acc[I][Jt][r] + d)), vr, 0);
                }
        }
    }
}

// Per-block partial sums over rows (layout of k_grads_shplrnn):
//   [M*L dW1 (row-major) | L*M dW2 | L dh2 | M dA | M dh1]
// dW1 += lam relu(u)^T, dW2 += delta z~^T with delta = (W1^T lam) * m, dh2 += delta, dA += lam * z~,
// dh1 += lam.  Each thread owns up to GB_PER entries of dW1 and of dW2 in registers.
constexpr int GB_PER = 32;

__global__ __launch_bounds__(256) void k_grads_big(const ShArgs a, const float *__restrict__ z,
                                                   const float *__restrict__ lam, const uint32_t *__restrict__ masks,
                                                   float *__restrict__ part) {
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, tid = threadIdx.x;
    // W2 kept transposed ([M][L]) so that the lanes l of a read take consecutive words
    float *w1 = smem, *w2t = w1 + (size_t)M * L, *zt = w2t + (size_t)L * M, *lm = zt + BG, *ru = lm + BG,
          *dl = ru + L;
    for (int e = tid; e < M * L; e += 256) {
        w1[e] = a.W1[e];
        const int l = e / M, k = e % M;
        w2t[(size_t)k * L + l] = a.W2[e];
    }
    const int LW = (L + 31) / 32;
    float g1[GB_PER], g2[GB_PER];
    // the (row, column) of this thread's entries of dW1 and of dW2 in one word (7, 6, 6, 7 bits:
    // M <= 128, L < 64), so that no row divides
    uint32_t ix[GB_PER];
#pragma unroll
    for (int q = 0; q < GB_PER; ++q) {
        g1[q] = g2[q] = 0.f;
        const uint32_t e = (uint32_t)(tid + 256 * q);
        ix[q] = (e / L) | ((e % L) << 7) | ((e / M) << 13) | ((e % M) << 19);
    }
    float dh2 = 0.f, dA = 0.f, dh1 = 0.f;
    const long rows = (long)a.B * T;
    const long per = (rows + gridDim.x - 1) / gridDim.x;
    const long r0 = (long)blockIdx.x * per, r1 = r0 + per < rows ? r0 + per : rows;
    // the next row's z~, lambda and mask word are loaded while this row is summed
    float zn = 0.f, ln = 0.f;
    uint32_t mn = 0u;
    auto load_row = [&](long row) {
        const int b = (int)(row / T), s = (int)(row % T);
        if (tid < M) {
            zn = big_forced(a, z, b, s, tid);
            ln = lam[(size_t)row * M + tid];
        }
        if ((tid >> 2) < L) mn = masks[(size_t)row * LW + (tid >> 7)];   // the word of unit tid / 4
    };
    if (r0 < r1) load_row(r0);
    __syncthreads();
    for (long row = r0; row < r1; ++row) {
        if (tid < M) {
            zt[tid] = zn;
            lm[tid] = ln;
        }
        const uint32_t mw = mn;
        if (row + 1 < r1) load_row(row + 1);
        __syncthreads();
        {
            // four threads per hidden unit l (L < 64), each summing every fourth k, added across the
            // four lanes
            const int l = tid >> 2, p = tid & 3;
            float u = 0.f, d = 0.f;
            if (l < L)
                for (int k = p; k < M; k += 4) {
                    u = fmaf(w2t[(size_t)k * L + l], zt[k], u);
                    d = fmaf(w1[(size_t)k * L + l], lm[k], d);
                }
            u += __shfl_xor(u, 1, 64);
            u += __shfl_xor(u, 2, 64);
            d += __shfl_xor(d, 1, 64);
            d += __shfl_xor(d, 2, 64);
            if (l < L && p == 0) {
                const bool m = (mw >> (l & 31)) & 1u;
                ru[l] = m ? u + (a.h2 ? a.h2[l] : 0.f) : 0.f;
                dl[l] = m ? d : 0.f;
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < GB_PER; ++q) {
            const int e = tid + 256 * q;
            if (e < M * L) {
                uint32_t x = ix[q];
                asm volatile("" : "+v"(x));   // keeps the packed word, not 4 hoisted LDS addresses, live
                g1[q] = fmaf(lm[x & 127u], ru[(x >> 7) & 63u], g1[q]);      // dW1[i][l]
                g2[q] = fmaf(dl[(x >> 13) & 63u], zt[(x >> 19) & 127u], g2[q]);   // dW2[l][j]
            }
        }
        if (tid < L) dh2 += dl[tid];
        if (tid < M) {
            dA = fmaf(lm[tid], zt[tid], dA);
            dh1 += lm[tid];
        }
        __syncthreads();
    }
    const size_t stride = (size_t)2 * M * L + L + 2 * M;
    float *pp = part + (size_t)blockIdx.x * stride;
#pragma unroll
    for (int q = 0; q < GB_PER; ++q) {
        const int e = tid + 256 * q;
        if (e < M * L) {
            pp[e] = g1[q];
            pp[(size_t)M * L + e] = g2[q];
        }
    }
    if (tid < L) pp[(size_t)2 * M * L + tid] = dh2;
    if (tid < M) {
        pp[(size_t)2 * M * L + L + tid] = dA;
        pp[(size_t)2 * M * L + L + M + tid] = dh1;
    }
}

// ---- host launchers (called by the dispatchers of the M <= 64 kernels when the padded width is
// 128) ------------------------------------------------------------------------------------------

int launch_chunk_product_big(bool rev, bool flip, int B, int T, int M, const float *J, const float *rhs,
                             float rhs_sign, float *P, float *v, const int *active, int C, int ncs, hipStream_t st) {
    const int grid = B * ncs;
    KTimer kt("k_chunk_product_dense", st);
#define CPB(R, F) \
    hipLaunchKernelGGL((k_chunk_product_big<R, F>), dim3(grid), dim3(256), 0, st, J, rhs, rhs_sign, P, v, active, B, T, M, C, ncs)
    if (!rev) { if (flip) CPB(false, true); else CPB(false, false); }
    else { if (flip) CPB(true, true); else CPB(true, false); }
#undef CPB
    DEER_LAUNCH_CHECK("k_chunk_product_big");
    return DEER_OK;
}

int launch_carry_big(bool rev, const float *P, const float *v, float *carry_in, const int *active, int B, int ncs,
                     int G, float *gws, hipStream_t st) {
    KTimer kt("k_carry", st);
    if (!G) {
        if (rev) hipLaunchKernelGGL(k_carry_big<true>, dim3(B), dim3(256), 0, st, P, v, carry_in, active, ncs, ncs, nullptr);
        else hipLaunchKernelGGL(k_carry_big<false>, dim3(B), dim3(256), 0, st, P, v, carry_in, active, ncs, ncs, nullptr);
        DEER_LAUNCH_CHECK("k_carry_big");
        return DEER_OK;
    }
    // workspace: group maps [B][ng][BG][BG], their walks from zero [B][ng][BG], group carries
    const int ng = (ncs + G - 1) / G;
    float *gq = gws;
    float *gu = gq + (size_t)B * ng * BG * BG;
    float *gc = gu + (size_t)B * ng * BG;
    const int grid = B * ng;
    if (rev) hipLaunchKernelGGL(k_carry_group_big<true>, dim3(grid), dim3(256), 0, st, P, v, gq, gu, active, ncs, G);
    else hipLaunchKernelGGL(k_carry_group_big<false>, dim3(grid), dim3(256), 0, st, P, v, gq, gu, active, ncs, G);
    DEER_LAUNCH_CHECK("k_carry_group_big");
    hipLaunchKernelGGL(k_carry_big<false>, dim3(B), dim3(256), 0, st, gq, gu, gc, active, ng, ng, nullptr);
    DEER_LAUNCH_CHECK("k_carry_big");
    if (rev) hipLaunchKernelGGL(k_carry_big<true>, dim3(grid), dim3(256), 0, st, P, v, carry_in, active, ncs, G, gc);
    else hipLaunchKernelGGL(k_carry_big<false>, dim3(grid), dim3(256), 0, st, P, v, carry_in, active, ncs, G, gc);
    DEER_LAUNCH_CHECK("k_carry_big");
    return DEER_OK;
}

int launch_fixup_big(int mode, bool flip, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                     const float *carry_in, float *z, float *out, const int *zsel, uint32_t *chain_bits,
                     const int *active, int C, int ncs, hipStream_t st) {
    const int grid = B * ncs;
    KTimer kt(mode == 2 ? "k_fixup_dense_rev" : "k_fixup_dense_fwd", st);
#define FXB(MO, F)                                                                                                  \
    hipLaunchKernelGGL((k_fixup_big<MO, F>), dim3(grid), dim3(256), 0, st, J, rhs, rhs_sign, carry_in, z, out, zsel, \
                       chain_bits, active, B, T, M, C, ncs)
    if (mode == 0) FXB(0, false);
    else if (mode == 1) { if (flip) FXB(1, true); else FXB(1, false); }
    else { if (flip) FXB(2, true); else FXB(2, false); }
#undef FXB
    DEER_LAUNCH_CHECK("k_fixup_big");
    return DEER_OK;
}

size_t big_resjac_lds(int M, int L) { return (size_t)2 * M * L * sizeof(float); }
size_t big_jacform_lds(int L) { return (size_t)2 * BG * ((L + 15) / 16 * 16) * sizeof(float); }
size_t big_grads_lds(int M, int L) { return ((size_t)2 * M * L + 2 * BG + 2 * L) * sizeof(float); }

int launch_resjac_big(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *F, float *r,
                      uint32_t *masks, const int *active, hipStream_t st) {
    // four rows per block; as many blocks as the LDS of the 256 CUs holds (160 KiB each, at most 8)
    const long rows = (long)a.B * a.T, want = (rows + 3) / 4;
    long per_cu = (long)(160 * 1024) / (long)big_resjac_lds(a.M, a.L);
    per_cu = per_cu < 1 ? 1 : (per_cu > 8 ? 8 : per_cu);
    const int grid = (int)(want < 256 * per_cu ? want : 256 * per_cu);
    KTimer kt("k_resjac_shplrnn", st);
    hipLaunchKernelGGL(k_resjac_big, dim3(grid), dim3(256), big_resjac_lds(a.M, a.L), st, a, z, zalt, zsel, F, r,
                       masks, active);
    DEER_LAUNCH_CHECK("k_resjac_big");
    return DEER_OK;
}

int launch_jacform_big(const ShArgs &a, const uint32_t *masks, float *J, const int *active, const float *gamma,
                       hipStream_t st) {
    // every block walks rows with W1 and V staged once: as many blocks as the LDS holds (two per CU
    // at L > 48)
    const long rows = (long)a.B * (a.t_hi > a.t_lo ? a.t_hi - a.t_lo : a.T);
    long per_cu = (long)(160 * 1024) / (long)big_jacform_lds(a.L);
    per_cu = per_cu < 1 ? 1 : (per_cu > 8 ? 8 : per_cu);
    const int grid = (int)(rows < 256 * per_cu ? rows : 256 * per_cu);
    const int LP = (a.L + 15) / 16 * 16;
    KTimer kt("k_jacform_shplrnn", st);
    if ((a.M & 3) == 0)
        hipLaunchKernelGGL(k_jacform_big<true>, dim3(grid), dim3(256), big_jacform_lds(a.L), st, a, masks, J, active, gamma, LP);
    else
        hipLaunchKernelGGL(k_jacform_big<false>, dim3(grid), dim3(256), big_jacform_lds(a.L), st, a, masks, J, active, gamma, LP);
    DEER_LAUNCH_CHECK("k_jacform_big");
    return DEER_OK;
}

int launch_grads_big(const ShArgs &a, const float *z, const float *lam, const uint32_t *masks, float *part, int nb,
                     hipStream_t st) {
    KTimer kt("k_grads_shplrnn", st);
    hipLaunchKernelGGL(k_grads_big, dim3(nb), dim3(256), big_grads_lds(a.M, a.L), st, a, z, lam, masks, part);
    DEER_LAUNCH_CHECK("k_grads_big");
    return DEER_OK;
}

}  // namespace deer
