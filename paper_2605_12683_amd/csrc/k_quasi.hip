// Quasi-DEER for the vanilla PLRNN: the GTF-DEER Newton update and backward recursion with
// every forced Jacobian J~_t replaced by its diagonal (the diagonal approximation the paper
// discusses with eq. DEER_update, and the quasi form of the backward recursion in the
// gradients appendix):
//   forward   Delta_t = d_t * Delta_{t-1} - r_t,        Delta_0 = 0
//   reverse   lam_{t-1} = d_t * lam_t + g_{t-1},        lam_T = g_T
//   d_t[i]  = (A_i + W_ii 1[z~_{t-1,i} > 0]) p_i,   p = 1 - a (the forcing projector)
// Every latent is then an independent first-order recurrence with a coefficient that varies
// in time, evaluated by a chunked scan: chunk aggregates (prod d, local solution from zero),
// a float64 carry pass over the chunks of a sequence, and a re-walk of every chunk from its
// carry.  Array index s holds step s + 1: coef[s] = d_{s+1}, taken at z~_s.
//
//   k_qdeer_resdiag   r (forward) and gamma_b d at every (b, s), from the current iterate
//   k_qdeer_chunk     (prod d, local solution) per (chain, latent)
//   k_qdeer_carry     carry entering every chunk of a sequence (two levels, float64)
//   k_qdeer_fixup     forward: z + Delta to the other iterate buffer, per-chain max|Delta| and
//                     max|z|; reverse: lam (optional) and the gradient partial sums of the
//                     chain, dW_ij += lam_i relu(z~_j), dA_i += lam_i z~_i, dh_i += lam_i
//   k_qdeer_pass      the adaptive loop's pass in one kernel: the fix-up of one update and the
//                     chunk aggregates of the next, with the pass-end control
//
// Lanes: a wave holds 64 / MP chains of MP lanes (lane = latent), MP in {16, 32, 64}; the
// ReLU row of a step goes through LDS when the lanes of a chain need each other's values.
#include "common.h"
#include "launch.h"
#include "newton_ctl.h"
#include "row16.h"

namespace deer {

namespace {
__device__ __forceinline__ float q_p(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

// sum_k row[k] * v[k] over the MP values of chain group n in LDS (two partial sums)
template <int MP>
__device__ __forceinline__ float q_dot(const float *lds, int n, const float *row) {
    const float4 *l4 = reinterpret_cast<const float4 *>(lds + n * MP);
    float a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int q = 0; q < MP / 4; ++q) {
        const float4 v = l4[q];
        a0 = fmaf(row[4 * q + 0], v.x, a0);
        a1 = fmaf(row[4 * q + 1], v.y, a1);
        a0 = fmaf(row[4 * q + 2], v.z, a0);
        a1 = fmaf(row[4 * q + 3], v.w, a1);
    }
    return a0 + a1;
}

// coefficient d of step s + 1 from the forced input z~_s, scaled by the damping g
__device__ __forceinline__ float q_coef(float zt, float Ai, float Wii, float pi, float g) {
    const float dj = zt > 0.f ? __fadd_rn(Ai, Wii) : Ai;
    return __fmul_rn(g, __fmul_rn(dj, pi));
}
}  // namespace

// ---------------------------------------------------------------------------------------
// r_s = z_s - F(z~_s) and coef_s = gamma_b d_{s+1} for every step s of sequence b =
// blockIdx.y, at its current iterate (zsel); a converged sequence's blocks exit at once.
// REV: coef only (the adjoint's right-hand side is the caller's cotangent or the MSE seed,
// formed in the scan kernels).  A wave takes NG x (64 / MP) consecutive steps per iteration
// (lane = latent) and loads the next iteration's inputs before it works on the current one.
// z~ is formed as everywhere else: fl(fl(p z) + fl(alpha x)) on the forced latents.
// ---------------------------------------------------------------------------------------
template <int MP, bool REV>
__global__ __launch_bounds__(64) void k_qdeer_resdiag(const float *__restrict__ A, const float *__restrict__ W,
                                                      const float *__restrict__ h, float alpha, int N,
                                                      const float *__restrict__ x, const float *__restrict__ z0,
                                                      const float *zbuf, const float *zalt, const int *__restrict__ zsel,
                                                      const int *__restrict__ active, const float *__restrict__ gamma,
                                                      float *__restrict__ rhs, float *__restrict__ coef, int B, int T,
                                                      int M, int tw) {
    constexpr int NCH = 64 / MP;
    constexpr int NG = 4;             // row groups per iteration (memory parallelism)
    constexpr int RS = NCH * NG;      // steps per iteration
    __shared__ __align__(16) float lds[NG][64];
    const int b = blockIdx.y;
    if (active && !active[b]) return;
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const bool iok = i < M;
    float wrow[MP];
#pragma unroll
    for (int j = 0; j < MP; ++j) wrow[j] = (!REV && iok && j < M) ? W[i * M + j] : 0.f;
    const float Ai = iok ? A[i] : 0.f;
    const float Wii = iok ? W[i * M + i] : 0.f;
    const float hi = (h && iok) ? h[i] : 0.f;
    const float pi = q_p(i, N, alpha);
    const float gmb = gamma ? gamma[b] : 1.f;
    const bool forced = i < N;
    const float *zs = cur_iter(zbuf, zalt, zsel, b) + (size_t)b * T * M;
    const float *xs = x + (size_t)b * (T + 1) * N;
    const float *zst = zs + i;
    float *cs = coef + (size_t)b * T * M + i;
    float *rs = REV ? nullptr : rhs + (size_t)b * T * M + i;
    const float zinit = !iok ? 0.f : (z0 ? z0[(size_t)b * M + i] : (forced ? xs[i] : 0.f));
    // inputs of the steps of one iteration: z_{s-1}, x_s (forced latents), z_s (residual)
    float zp[NG], xq[NG], zv[NG];
    auto load = [&](int sb) {
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int s = sb + q * NCH + n;
            const bool ok = s < T && iok;
            zp[q] = (ok && s > 0) ? zst[(size_t)(s - 1) * M] : 0.f;
            xq[q] = (ok && s > 0 && forced) ? xs[(size_t)s * N + i] : 0.f;
            zv[q] = (ok && !REV) ? zst[(size_t)s * M] : 0.f;
        }
    };
    const int stride = gridDim.x * RS;
    int sb = blockIdx.x * RS;
    load(sb);
    for (; sb < T; sb += stride) {
        float zt[NG], zc[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int s = sb + q * NCH + n;
            // latent warm-up (s <= tw): the observed latents take the data (alpha_s = 1)
            zt[q] = s == 0 ? zinit
                           : (forced ? (s <= tw ? xq[q] : __fadd_rn(__fmul_rn(pi, zp[q]), __fmul_rn(alpha, xq[q])))
                                     : zp[q]);
            zc[q] = zv[q];
        }
        load(sb + stride);   // the next iteration's inputs, in flight during this one
        float F[NG];
        if (!REV) {
#pragma unroll
            for (int q = 0; q < NG; ++q) lds[q][lane] = zt[q] > 0.f ? zt[q] : 0.f;
            lds_barrier();
#pragma unroll
            for (int q = 0; q < NG; ++q) {
                F[q] = fmaf(Ai, zt[q], q_dot<MP>(lds[q], n, wrow)) + hi;
                __builtin_amdgcn_sched_barrier(0);
            }
            lds_barrier();
        }
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int s = sb + q * NCH + n;
            if (s < T && iok) {
                cs[(size_t)s * M] = q_coef(zt[q], Ai, Wii, (forced && s <= tw) ? 0.f : pi, gmb);   // P_1
                if (!REV) rs[(size_t)s * M] = zc[q] - F[q];
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// Chunk aggregates.  Chain id = b ncs + c covers array indices [s0, s1), s0 = c C.
//   forward: y_s = coef_s y_{s-1} + sgn rhs_s from y_{s0-1} = 0; P = prod coef_s, v = y_{s1-1}
//   reverse: y_s = coef_{s+1} y_{s+1} + g_s from y_{s1} = 0 (coef_T = 0);
//            P = prod coef_{s+1}, v = y_{s0};  g = rhs, or the MSE seed
//            seed_scale (z_s - x_{s+1}) on the first N latents when rhs is null
// Loads are issued QB steps at a time (indices clamped to the chain) before they are used.
// ---------------------------------------------------------------------------------------
constexpr int QB = 8;

template <int MP, bool REV>
__global__ __launch_bounds__(64) void k_qdeer_chunk(const float *__restrict__ coef, const float *__restrict__ rhs,
                                                    float sgn, const float *__restrict__ z, const float *__restrict__ x,
                                                    float seed_scale, int N, const int *__restrict__ active,
                                                    float *__restrict__ Pout, float *__restrict__ vout, int B, int T,
                                                    int M, int C, int ncs, int tw) {
    constexpr int NCH = 64 / MP;
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * NCH + n;
    const bool ok = id < B * ncs && i < M;
    const int b = ok ? id / ncs : 0, c = ok ? id % ncs : 0;
    if (!ok || (active && !active[b])) return;
    const int s0 = c * C, s1 = min(s0 + C, T);
    const size_t base = (size_t)b * T;
    float P = 1.f, y = 0.f;
    for (int k0 = 0; k0 < s1 - s0; k0 += QB) {
        float cv[QB], gv[QB];
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            const int kk = min(k0 + k, s1 - s0 - 1);
            const int s = REV ? s1 - 1 - kk : s0 + kk;
            const int sc = REV ? s + 1 : s;
            cv[k] = sc < T ? coef[(base + sc) * M + i] : 0.f;
            if (rhs) {
                gv[k] = rhs[(base + s) * M + i];
            } else {
                gv[k] = (i < N && s >= tw) ? __fmul_rn(seed_scale, __fsub_rn(z[(base + s) * M + i],
                                                                                x[((size_t)b * (T + 1) + s + 1) * N + i]))
                                           : 0.f;   // no MSE seed for the warm-up states s < tw
            }
        }
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            if (k0 + k < s1 - s0) {
                y = fmaf(cv[k], y, sgn * gv[k]);
                P = P * cv[k];
            }
        }
    }
    Pout[(size_t)id * MP + i] = P;
    vout[(size_t)id * MP + i] = y;
}

// ---------------------------------------------------------------------------------------
// Carries: block = sequence, threads = (group gq of CG consecutive chunks in processing
// order, latent i).  X_0 = 0 and X_{l+1} = P_l X_l + v_l over the chunks l in processing
// order (forward: c = l; reverse: c = ncs - 1 - l); carry[c] = X_l.  Group maps composed in
// float64, a serial pass over the groups, every group re-walked from its carry.
// ---------------------------------------------------------------------------------------
template <int MP, bool REV>
__global__ __launch_bounds__(1024) void k_qdeer_carry(const float *__restrict__ P, const float *__restrict__ v,
                                                      float *__restrict__ carry, const int *__restrict__ active, int M,
                                                      int ncs) {
    constexpr int NGQ = 1024 / MP;
    __shared__ double gp[NGQ][MP], gv[NGQ][MP];
    const int b = blockIdx.x;
    if (active && !active[b]) return;
    const int i = threadIdx.x % MP, gq = threadIdx.x / MP;
    const int CG = (ncs + NGQ - 1) / NGQ;
    const int l0 = min(gq * CG, ncs), l1 = min(l0 + CG, ncs);
    const size_t cb = (size_t)b * ncs;
    auto chunk_of = [&](int l) { return REV ? ncs - 1 - l : l; };
    double ap = 1.0, av = 0.0;
    if (i < M) {
        for (int l = l0; l < l1; l += QB) {
            float pq[QB], vq[QB];
#pragma unroll
            for (int k = 0; k < QB; ++k) {
                const size_t e = (cb + chunk_of(min(l + k, l1 - 1))) * MP + i;
                pq[k] = P[e];
                vq[k] = v[e];
            }
#pragma unroll
            for (int k = 0; k < QB; ++k) {
                if (l + k < l1) {
                    av = (double)pq[k] * av + (double)vq[k];
                    ap = (double)pq[k] * ap;
                }
            }
        }
    }
    gp[gq][i] = ap;
    gv[gq][i] = av;
    __syncthreads();
    if (gq == 0 && i < M) {
        double X = 0.0;
        for (int g2 = 0; g2 < NGQ; ++g2) {
            const double xp = gp[g2][i], xv = gv[g2][i];
            gv[g2][i] = X;
            X = xp * X + xv;
        }
    }
    __syncthreads();
    if (i >= M) return;
    double X = gv[gq][i];
    for (int l = l0; l < l1; l += QB) {
        float pq[QB], vq[QB];
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            const size_t e = (cb + chunk_of(min(l + k, l1 - 1))) * MP + i;
            pq[k] = P[e];
            vq[k] = v[e];
        }
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            if (l + k < l1) {
                carry[(cb + chunk_of(l + k)) * MP + i] = (float)X;
                X = (double)pq[k] * X + (double)vq[k];
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// Forward fix-up: Delta from the carry, the next iterate z + Delta written to the other
// buffer, per-chain max|Delta| and max|z| bits (reduced per sequence by k_seq_ctl).
// ---------------------------------------------------------------------------------------
template <int MP>
__global__ __launch_bounds__(64) void k_qdeer_fixup_fwd(const float *__restrict__ coef, const float *__restrict__ rhs,
                                                        const float *__restrict__ carry, float *zbuf, float *zalt,
                                                        const int *__restrict__ zsel, uint32_t *__restrict__ chain_bits,
                                                        const int *__restrict__ active, int B, int T, int M, int C,
                                                        int ncs) {
    constexpr int NCH = 64 / MP;
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * NCH + n;
    const bool in = id < B * ncs;
    const int b = in ? id / ncs : 0, c = in ? id % ncs : 0;
    const bool ok = in && (!active || active[b]);
    const bool run = ok && i < M;
    const int s0 = c * C, s1 = ok ? min(s0 + C, T) : s0;
    const size_t base = (size_t)b * T;
    const float *zin = cur_iter(zbuf, zalt, zsel, b);
    float *zout = next_iter(zbuf, zalt, zsel, b);
    float D = run ? carry[(size_t)id * MP + i] : 0.f;
    uint32_t emax = 0u, zmax = 0u;
    for (int k0 = 0; k0 < s1 - s0; k0 += QB) {
        float cv[QB], rv[QB], zv[QB];
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            const size_t e = (base + s0 + min(k0 + k, s1 - s0 - 1)) * M + i;
            cv[k] = run ? coef[e] : 0.f;
            rv[k] = run ? rhs[e] : 0.f;
            zv[k] = run ? zin[e] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < QB; ++k) {
            if (run && k0 + k < s1 - s0) {
                D = fmaf(cv[k], D, -rv[k]);
                zout[(base + s0 + k0 + k) * M + i] = zv[k] + D;
                const uint32_t ab = abs_bits(D), zb = abs_bits(zv[k]);
                emax = emax > ab ? emax : ab;
                zmax = zmax > zb ? zmax : zb;
            }
        }
    }
#pragma unroll
    for (int off = MP / 2; off > 0; off >>= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
        const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
        emax = emax > o ? emax : o;
        zmax = zmax > oz ? zmax : oz;
    }
    if (ok && i == 0) {
        chain_bits[id] = emax;
        chain_bits[(size_t)B * ncs + id] = zmax;
    }
}

// ---------------------------------------------------------------------------------------
// One kernel per pass of the adaptive loop.  A block takes a group of GS = QF_WPB (64 / MP)
// consecutive chunks of one sequence (the chunk count per sequence is padded to a multiple of
// GS with empty chunks) and runs, per chunk:
//   1. when the sequence's aggregates of the previous kernel belong to its current iterate
//      (nd.pv == pass_no): the chunk's carry, walked in float64 over the group maps of the
//      groups before it and the chunk aggregates before it in its group, then the fix-up
//      Delta_s = coef_s Delta_{s-1} - r_s with r and coef formed again from z and x by the
//      operations step 2 of the previous kernel formed them with (so they are the values its
//      aggregates hold), z + Delta written to the other iterate buffer;
//   2. the chunk aggregates of the next update at the new iterate (or at the current one when
//      step 1 did not run): prod coef and the local solution from zero, with the damping that
//      an accepted update leads to, and the group map of the block (float64);
//   3. the pass-end control of step 1's update (seq_arrive), which also records in nd.pv that
//      the aggregates just formed belong to the accepted iterate.
// Step 2 at a chunk's first step needs the new iterate at the step before the chunk: that is
// z + carry, and the chunk before puts exactly that value there (it forms this chunk's carry
// with the same float64 operations on the same operands instead of taking the end of its own
// recurrence), so no wave waits for another.  Aggregates alternate between two buffers.
// ---------------------------------------------------------------------------------------
// Products (W relu(zt_q))_i for the TS steps q of a tile, lane = latent i of its chain.  MP = 16:
// formed here by DPP row rotations into dq (w: the row's weights in rotation order); else the
// ReLU rows go to the wave's LDS rows, and q_tile_dot reads product q where it is consumed (all
// of them at once would hold every operand in registers).
template <int MP, int TS>
__device__ __forceinline__ void q_tile_rows(const float (&zt)[TS], const float (&w)[MP], float (*lr)[64], int lane,
                                            float (&dq)[TS]) {
    if constexpr (MP == 16) {
#pragma unroll
        for (int q = 0; q < TS; q += 2)
            row16_dot2(w, zt[q] > 0.f ? zt[q] : 0.f, zt[q + 1] > 0.f ? zt[q + 1] : 0.f, dq[q], dq[q + 1]);
    } else {
#pragma unroll
        for (int q = 0; q < TS; ++q) lr[q][lane] = zt[q] > 0.f ? zt[q] : 0.f;
        wave_lds_sync();
    }
}
template <int MP, int TS>
__device__ __forceinline__ float q_tile_dot(const float (&dq)[TS], const float (&w)[MP], float (*lr)[64], int n, int q) {
    if constexpr (MP == 16) return dq[q];
    else return q_dot<MP>(lr[q], n, w);
}

constexpr int QF_WPB = 8;   // waves per block
constexpr int QF_TS = 8;    // steps per tile
constexpr int QF_MAXG = 32; // groups per sequence at most

template <int MP>
__global__ __launch_bounds__(64 * QF_WPB) void k_qdeer_pass(
    const float *__restrict__ A, const float *__restrict__ W, const float *__restrict__ h, float alpha, int N,
    const float *__restrict__ x, const float *__restrict__ z0, float *zbuf, float *zalt, int T, int M, int C, int ncs,
    const float *__restrict__ Pin, const float *__restrict__ vin, const double *__restrict__ gin,
    float *__restrict__ Pout, float *__restrict__ vout, double *__restrict__ gout, FusedCtl fc, uint32_t *mark,
    uint32_t pass_no, int tw) {
    constexpr int NCH = 64 / MP, GS = QF_WPB * NCH, TS = QF_TS;
    __shared__ __align__(16) float rl[MP == 16 ? 1 : QF_WPB][TS][64];   // ReLU rows of a tile, per wave (MP > 16)
    __shared__ float sW[MP * MP];
    __shared__ float sag[2][GS][MP];                      // the previous kernel's chunk aggregates of the group
    __shared__ float sagn[2][GS][MP];                     // the next update's
    __shared__ double sG[2][QF_MAXG][MP];                 // group maps of the groups up to this one
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, n = lane / MP, i = lane % MP;
    if (mark && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(mark, pass_no, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const NewtonDev &nd = fc.nd;
    const int ngm = ncs / GS;
    const int b = blockIdx.x / ngm, grp = blockIdx.x - b * ngm;
    if (nd.act[b] == 0) return;   // the whole block
    const bool have = nd.pv[b] == pass_no;
    const int sel = nd.sel[b];
    const float gam = nd.gamma[b];
    float omn = nd.om[b];   // the damping of the next update if this one is kept
    if (omn > 0.f) omn = omn / fc.dp.shrink < fc.dp.floor ? 0.f : omn / fc.dp.shrink;
    const float gnext = have ? 1.f - omn : gam;
    const float *const zc = sel ? zalt : zbuf;   // current iterate
    float *const zn = sel ? zbuf : zalt;         // the update's output
    const int kg = wv * NCH + n;                 // this lane's chunk within the group
    const int c = grp * GS + kg;
    const int s0 = c * C;
    const int len = max(min(s0 + C, T) - s0, 0);  // 0: a padding chunk
    int maxlen = len;                              // the wave's tile loop is uniform
#pragma unroll
    for (int off = 32; off >= MP; off >>= 1) maxlen = max(maxlen, __shfl_xor(maxlen, off, 64));
    const bool iok = i < M, forced = i < N;
    const size_t zrow = (size_t)b * T;
    const float *xs = x + (size_t)b * (T + 1) * N;
    // buffer resources over the sequence's rows (a load past its end reads zero): a lane's byte
    // offset is that of its chunk's first step, a tile step adds a wave-uniform offset
    const auto rzc = bounded_rsrc(zc + zrow * M, (uint32_t)T * M * 4u);
    const auto rzn = bounded_rsrc(zn + zrow * M, (uint32_t)T * M * 4u);
    const auto rx = bounded_rsrc(xs, (uint32_t)(T + 1) * N * 4u);
    const uint32_t vz = (iok && len > 0) ? 4u * ((uint32_t)s0 * M + i) : kOffLane;
    const uint32_t vx = (forced && len > 0) ? 4u * ((uint32_t)s0 * N + i) : kOffLane;
    // the first tile's inputs and z_{s0-1} of the current iterate (the initial state at s0 = 0,
    // taken as the forced state) go out first
    float zq[TS], xq[TS];
    auto load = [&](int t0) {
#pragma unroll
        for (int q = 0; q < TS; ++q) {
            zq[q] = bload(rzc, vz, 4 * (t0 + q) * M);
            xq[q] = bload(rx, vx, 4 * (t0 + q) * N);
        }
    };
    load(0);
    float zprev = 0.f;
    if (iok && len > 0) {
        if (s0 == 0) zprev = z0 ? z0[(size_t)b * M + i] : (forced ? xs[i] : 0.f);
        else zprev = zc[(zrow + s0 - 1) * M + i];
    }
    // weights, and the previous kernel's aggregates this block walks, through LDS
    for (int t = threadIdx.x; t < M * M; t += 64 * QF_WPB) sW[t] = W[t];
    if (have) {
        const float *Pg = Pin + ((size_t)b * ncs + (size_t)grp * GS) * MP;
        const float *vg = vin + ((size_t)b * ncs + (size_t)grp * GS) * MP;
        for (int t = threadIdx.x; t < GS * MP; t += 64 * QF_WPB) {
            sag[0][t / MP][t % MP] = Pg[t];
            sag[1][t / MP][t % MP] = vg[t];
        }
        const double *G = gin + (size_t)b * ngm * 2 * MP;
        for (int t = threadIdx.x; t < (grp + 1) * MP; t += 64 * QF_WPB) {   // groups 0 .. grp
            const int q = t / MP, j = t % MP;
            sG[0][q][j] = G[(size_t)q * 2 * MP + j];
            sG[1][q][j] = G[(size_t)q * 2 * MP + MP + j];
        }
    }
    __syncthreads();
    float wrow[MP];   // row i of W (MP = 16: in the order of the row rotations)
    if constexpr (MP == 16) {
        int src[16];
        row_sources(i, src);
#pragma unroll
        for (int k = 0; k < 16; ++k) wrow[k] = (iok && src[k] < M) ? sW[i * M + src[k]] : 0.f;
    } else {
#pragma unroll
        for (int j = 0; j < MP; ++j) wrow[j] = (iok && j < M) ? sW[i * M + j] : 0.f;
    }
    const float Ai = iok ? A[i] : 0.f, Wii = iok ? sW[i * M + i] : 0.f, hi = (h && iok) ? h[i] : 0.f;
    const float pi = q_p(i, N, alpha);
    // ---- the chunk's carry and the next chunk's (float64 walks over the group maps before the
    // group and the chunk aggregates before the chunk) ----
    float D = 0.f, Dn = 0.f;
    const bool usenext = have && s0 + C < T;   // the next chunk holds steps
    if (have && iok) {
        // operands read 8 at a time ahead of the dependent multiply-adds
        double X = 0.0;
        for (int q0 = 0; q0 < grp; q0 += 8) {
            double gp[8], gv[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int q = min(q0 + k, grp - 1);
                gp[k] = sG[0][q][i];
                gv[k] = sG[1][q][i];
            }
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (q0 + k < grp) X = fma(gp[k], X, gv[k]);
        }
        const double Xg = X;
        for (int k0 = 0; k0 < kg; k0 += 8) {
            float pp[8], vv[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int q = min(k0 + k, kg - 1);
                pp[k] = sag[0][q][i];
                vv[k] = sag[1][q][i];
            }
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (k0 + k < kg) X = fma((double)pp[k], X, (double)vv[k]);
        }
        D = (float)X;
        if (usenext) {   // the operations the next chunk forms its carry with
            const double Xn = kg + 1 == GS ? fma(sG[0][grp][i], Xg, sG[1][grp][i])
                                           : fma((double)sag[0][kg][i], X, (double)sag[1][kg][i]);
            Dn = (float)Xn;
        }
    }
    // z_{s0-1} of the iterate the next update is formed at (as the chunk before stores it)
    float zpn = have ? zprev + D : zprev;
    uint32_t emax = 0u, zmax = 0u;
    float u = 0.f, Pn = 1.f;
    float (*const lr)[64] = rl[MP == 16 ? 0 : wv];
    // Branch-free tile bodies (the DPP products need every lane): a lane past its chunk's end
    // keeps its recurrences and stores nothing; padding lanes (i >= M) read zeros, so their
    // residuals, coefficients and Delta are zero.
    for (int t0 = 0; t0 < maxlen; t0 += TS) {
        float zv[TS], xv[TS];
#pragma unroll
        for (int q = 0; q < TS; ++q) {
            zv[q] = zq[q];
            xv[q] = xq[q];
        }
        if (t0 + TS < maxlen) load(t0 + TS);   // the next tile's inputs, in flight during this one
        if (have) {
            // residual and coefficients at the current iterate, then the fix-up
            float zt[TS];
#pragma unroll
            for (int q = 0; q < TS; ++q) {
                const int s = s0 + t0 + q;
                const float fz = s <= tw ? xv[q] : __fadd_rn(__fmul_rn(pi, zprev), __fmul_rn(alpha, xv[q]));
                zt[q] = (s == 0 || !forced) ? zprev : fz;
                zprev = zv[q];
            }
            float dq[TS];
            q_tile_rows<MP, TS>(zt, wrow, lr, lane, dq);
#pragma unroll
            for (int q = 0; q < TS; ++q) {
                const int s = s0 + t0 + q;
                const float F = fmaf(Ai, zt[q], q_tile_dot<MP, TS>(dq, wrow, lr, n, q)) + hi;
                const float r = zv[q] - F;
                const float cf = q_coef(zt[q], Ai, Wii, (forced && s <= tw) ? 0.f : pi, gam);
                const bool st = t0 + q < len;
                const float Dq = fmaf(cf, D, -r);
                D = st ? Dq : D;
                const float dap = (usenext && t0 + q == len - 1) ? Dn : D;
                const float znew = zv[q] + dap;
                bstore_u(rzn, __float_as_uint(znew), st ? vz : kOffLane, 4 * (t0 + q) * M);
                const uint32_t ab = st ? abs_bits(dap) : 0u, zb = st ? abs_bits(zv[q]) : 0u;
                emax = emax > ab ? emax : ab;
                zmax = zmax > zb ? zmax : zb;
                zv[q] = st ? znew : zv[q];
            }
            if constexpr (MP != 16) wave_lds_sync();   // the rows are read before they are rewritten
        }
        // the next update's residual and coefficients at the (new) iterate: chunk aggregates
        {
            float zt[TS];
#pragma unroll
            for (int q = 0; q < TS; ++q) {
                const int s = s0 + t0 + q;
                const float fz = s <= tw ? xv[q] : __fadd_rn(__fmul_rn(pi, zpn), __fmul_rn(alpha, xv[q]));
                zt[q] = (s == 0 || !forced) ? zpn : fz;
                zpn = zv[q];
            }
            float dq[TS];
            q_tile_rows<MP, TS>(zt, wrow, lr, lane, dq);
#pragma unroll
            for (int q = 0; q < TS; ++q) {
                const int s = s0 + t0 + q;
                const float F = fmaf(Ai, zt[q], q_tile_dot<MP, TS>(dq, wrow, lr, n, q)) + hi;
                const float r = zv[q] - F;
                const float cf = q_coef(zt[q], Ai, Wii, (forced && s <= tw) ? 0.f : pi, gnext);
                const bool st = t0 + q < len;
                const float uq = fmaf(cf, u, -r), pq = Pn * cf;
                u = st ? uq : u;
                Pn = st ? pq : Pn;
            }
            if constexpr (MP != 16) wave_lds_sync();
        }
    }
    if (!iok) {
        u = 0.f;
        Pn = 1.f;
    }
    __shared__ uint32_t smx[2][QF_WPB];
    if (have) {
        emax = wave_max_u32(emax);
        zmax = wave_max_u32(zmax);
        if (lane == 0) {
            smx[0][wv] = emax;
            smx[1][wv] = zmax;
        }
    }
    // ---- chunk aggregates of the next update ----
    const size_t e = ((size_t)b * ncs + c) * MP + i;
    Pout[e] = Pn;
    vout[e] = u;
    sagn[0][kg][i] = Pn;
    sagn[1][kg][i] = u;
    __syncthreads();
    // ---- pass-end control of the current update (once per block: its chunks share b) ----
    if (threadIdx.x == 0) {
        if (have) {
            uint32_t em = smx[0][0], zm = smx[1][0];
            for (int w = 1; w < QF_WPB; ++w) {
                em = em > smx[0][w] ? em : smx[0][w];
                zm = zm > smx[1][w] ? zm : smx[1][w];
            }
            seq_arrive(fc, b, GS, ncs, em, zm, pass_no + 1u);
        } else {
            // aggregates of the current iterate (nothing else of this sequence runs in this kernel)
            nd.pv[b] = pass_no + 1u;
        }
    }
    // ---- the group map of the next update ----
    if (threadIdx.x >= MP) return;
    double gp = 1.0, gv = 0.0;
    for (int k = 0; k < GS; ++k) {
        const double pk = (double)sagn[0][k][threadIdx.x];
        gv = fma(pk, gv, (double)sagn[1][k][threadIdx.x]);
        gp = gp * pk;
    }
    double *Go = gout + ((size_t)b * ngm + grp) * 2 * MP + threadIdx.x;
    Go[0] = gp;
    Go[MP] = gv;
}

// ---------------------------------------------------------------------------------------
// Reverse fix-up: lam from the carry (lam_{s1} of the chunk), walked down the chunk,
// optionally written, with the gradient partial sums of the chain at the forced inputs
// z~_s of the same trajectory (the ReLU row of every step through LDS):
//   gpart[id][i][j] (j < MP) = sum lam_i relu(z~_j),  [MP] = sum lam_i z~_i,  [MP+1] = sum lam_i
// ---------------------------------------------------------------------------------------
template <int MP, bool GR>
__global__ __launch_bounds__(64) void k_qdeer_fixup_rev(const float *__restrict__ coef, const float *__restrict__ g,
                                                        float seed_scale, float alpha, int N,
                                                        const float *__restrict__ x, const float *__restrict__ z0,
                                                        const float *__restrict__ z, const float *__restrict__ carry,
                                                        float *__restrict__ lam, float *__restrict__ gpart, int B,
                                                        int T, int M, int C, int ncs, int tw) {
    constexpr int NCH = 64 / MP;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * NCH + n;
    const bool in = id < B * ncs;
    const int b = in ? id / ncs : 0, c = in ? id % ncs : 0;
    const bool run = in && i < M;
    const int s0 = c * C, s1 = in ? min(s0 + C, T) : s0;
    // every chain of the wave takes the same number of steps (shorter ones idle), so the
    // LDS exchange is wave-uniform
    const int len = s1 - s0;
    int maxlen = len;
#pragma unroll
    for (int off = 32; off >= MP; off >>= 1) maxlen = max(maxlen, __shfl_xor(maxlen, off, 64));
    const size_t base = (size_t)b * T;
    float L = run ? carry[(size_t)id * MP + i] : 0.f;
    float gw[MP], ga = 0.f, gh = 0.f;
#pragma unroll
    for (int j = 0; j < MP; ++j) gw[j] = 0.f;
    for (int k = 0; k < maxlen; ++k) {
        const bool st = run && k < len;
        const int s = s1 - 1 - k;
        float cv = 0.f, gv = 0.f, zt = 0.f;
        if (st) {
            cv = s + 1 < T ? coef[(base + s + 1) * M + i] : 0.f;
            if (g) {
                gv = g[(base + s) * M + i];
            } else {
                gv = (i < N && s >= tw) ? __fmul_rn(seed_scale, __fsub_rn(z[(base + s) * M + i],
                                                                            x[((size_t)b * (T + 1) + s + 1) * N + i]))
                                        : 0.f;   // no MSE seed for the warm-up states s < tw
            }
            if (GR) zt = forced_state(x, z0, z, b, s, i, T, M, N, alpha, tw);
            L = fmaf(cv, L, gv);
            if (lam) lam[(base + s) * M + i] = L;
            ga = fmaf(L, zt, ga);
            gh += L;
        }
        if (!GR) continue;
        lds[lane] = (st && zt > 0.f) ? zt : 0.f;
        wave_lds_sync();
        const float4 *l4 = reinterpret_cast<const float4 *>(lds + n * MP);
        const float Ls = st ? L : 0.f;
#pragma unroll
        for (int q = 0; q < MP / 4; ++q) {
            const float4 v4 = l4[q];
            gw[4 * q + 0] = fmaf(Ls, v4.x, gw[4 * q + 0]);
            gw[4 * q + 1] = fmaf(Ls, v4.y, gw[4 * q + 1]);
            gw[4 * q + 2] = fmaf(Ls, v4.z, gw[4 * q + 2]);
            gw[4 * q + 3] = fmaf(Ls, v4.w, gw[4 * q + 3]);
        }
        wave_lds_sync();
    }
    if (!GR || !in) return;
    float *gp = gpart + ((size_t)id * MP + i) * (MP + 2);
#pragma unroll
    for (int j = 0; j < MP; ++j) gp[j] = gw[j];
    gp[MP] = ga;
    gp[MP + 1] = gh;
}

// ---------------------------------------------------------------------------------------
// Shallow PLRNN coefficients: coef_s[i] = gamma_b (A_i + sum_l W1_il m_{s,l} W2_li) p_i, the
// diagonal of J_F = diag(A) + W1 diag(m) W2 times P_alpha, from the hidden-unit ReLU masks of
// step s.  Block = (tile of steps, sequence b): C_il = W1_il W2_li in LDS, threads = (row,
// latent); a converged sequence's blocks exit at once.
// ---------------------------------------------------------------------------------------
constexpr int QSR = 256;   // threads per block

__global__ __launch_bounds__(QSR) void k_qdeer_shdiag(const float *__restrict__ A, const float *__restrict__ W1,
                                                     const float *__restrict__ W2, float alpha, int N,
                                                     const uint32_t *__restrict__ masks, const int *__restrict__ active,
                                                     const float *__restrict__ gamma, float *__restrict__ coef, int T,
                                                     int M, int L, int tw) {
    extern __shared__ float Cs[];   // [M][L]
    const int b = blockIdx.y;
    if (active && !active[b]) return;
    for (int e = threadIdx.x; e < M * L; e += QSR) {
        const int i = e / L, l = e % L;
        Cs[e] = W1[i * L + l] * W2[l * M + i];
    }
    __syncthreads();
    const int LW = (L + 31) / 32;
    const float gm = gamma ? gamma[b] : 1.f;
    const int rows = QSR / M;   // steps handled at once (M <= 64)
    const int r = threadIdx.x / M, i = threadIdx.x % M;
    if (r >= rows) return;
    const float Ai = A[i], pi = i < N ? __fsub_rn(1.0f, alpha) : 1.0f;
    const float *Ci = Cs + i * L;
    for (int s = blockIdx.x * rows + r; s < T; s += gridDim.x * rows) {
        const uint32_t *mw = masks + ((size_t)b * T + s) * LW;
        float d = 0.f;
        for (int w = 0; w < LW; ++w) {
            const uint32_t bits = mw[w];
            const float *cw = Ci + 32 * w;
            const int nb = min(32, L - 32 * w);
            for (int j = 0; j < nb; ++j)
                if ((bits >> j) & 1u) d += cw[j];
        }
        coef[((size_t)b * T + s) * M + i] = gm * ((Ai + d) * ((i < N && s <= tw) ? 0.f : pi));   // P_1 in the warm-up
    }
}

int launch_qdeer_shdiag(const ShArgs &a, const uint32_t *masks, const int *active, const float *gamma, float *coef,
                        hipStream_t st) {
    const int rows = QSR / a.M;
    long gx = (a.T + rows - 1) / rows;
    const long cap = (2048L + a.B - 1) / a.B;
    if (gx > cap) gx = cap;
    KTimer kt("k_qdeer_shdiag", st);
    hipLaunchKernelGGL(k_qdeer_shdiag, dim3((unsigned)gx, (unsigned)a.B), dim3(QSR), (size_t)a.M * a.L * sizeof(float),
                       st, a.A, a.W1, a.W2, a.alpha, a.N, masks, active, gamma, coef, a.T, a.M, a.L, a.tw);
    DEER_LAUNCH_CHECK("k_qdeer_shdiag");
    return DEER_OK;
}

// ---------------------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------------------
static int q_padded(int M) { return M <= 16 ? 16 : (M <= 32 ? 32 : 64); }

// chunk length: about 4096 waves of chains, at least 16 steps, at most 1024 chunks per
// sequence (the carry pass walks ncs / (1024 / MP) chunks per thread twice)
int qdeer_chunk_len(int B, int T, int M) {
    const int MP = q_padded(M);
    const long per_wave = 64 / MP;
    long C = 16;
    while (C < T && (long)B * ((T + C - 1) / C) > 4096 * per_wave) C *= 2;
    while ((T + C - 1) / C > 1024) C *= 2;
    return (int)(C < T ? C : (T > 0 ? T : 1));
}

// residual grid: y = sequence, x = tiles of 4 (64 / MP) steps, about 4096 blocks in all
static dim3 q_grid_rows(int B, int T, int MP) {
    const long tiles = (T + 4L * (64 / MP) - 1) / (4L * (64 / MP));
    long gx = (4096L + B - 1) / B;
    if (gx > tiles) gx = tiles;
    if (gx < 1) gx = 1;
    return dim3((unsigned)gx, (unsigned)B);
}

int launch_qdeer_update(const PlrnnArgs &a, float *z, float *zalt, const int *zsel, const int *active,
                        const float *gamma, float *rhs, float *coef, float *P, float *v, float *carry,
                        uint32_t *chain_bits, int C, int ncs, hipStream_t st) {
    const int MP = q_padded(a.M);
    {
        KTimer kt("k_qdeer_resdiag", st);
        const dim3 grid = q_grid_rows(a.B, a.T, MP);
#define RD(MPV) \
    hipLaunchKernelGGL((k_qdeer_resdiag<MPV, false>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x, a.z0, \
                       (const float *)z, (const float *)zalt, zsel, active, gamma, rhs, coef, a.B, a.T, a.M, a.tw)
        if (MP == 16) RD(16); else if (MP == 32) RD(32); else RD(64);
#undef RD
    }
    DEER_LAUNCH_CHECK("k_qdeer_resdiag");
    return launch_qdeer_scan_fwd(a.B, a.T, a.M, a.x, a.N, z, zalt, zsel, active, rhs, coef, P, v, carry, chain_bits, C,
                                 ncs, st);
}

int launch_qdeer_scan_fwd(int B, int T, int M, const float *x, int N, float *z, float *zalt, const int *zsel,
                          const int *active, const float *rhs, const float *coef, float *P, float *v, float *carry,
                          uint32_t *chain_bits, int C, int ncs, hipStream_t st) {
    const int MP = q_padded(M);
    const int nchains = B * ncs;
    const int gridc = (nchains + 64 / MP - 1) / (64 / MP);
    {
        KTimer kt("k_qdeer_chunk", st);
#define CK(MPV) \
    hipLaunchKernelGGL((k_qdeer_chunk<MPV, false>), dim3(gridc), dim3(64), 0, st, coef, rhs, -1.f, (const float *)nullptr, \
                       x, 0.f, N, active, P, v, B, T, M, C, ncs, 0)
        if (MP == 16) CK(16); else if (MP == 32) CK(32); else CK(64);
#undef CK
    }
    DEER_LAUNCH_CHECK("k_qdeer_chunk");
    {
        KTimer kt("k_qdeer_carry", st);
#define CR(MPV) \
    hipLaunchKernelGGL((k_qdeer_carry<MPV, false>), dim3(B), dim3(1024), 0, st, (const float *)P, (const float *)v, carry, \
                       active, M, ncs)
        if (MP == 16) CR(16); else if (MP == 32) CR(32); else CR(64);
#undef CR
    }
    DEER_LAUNCH_CHECK("k_qdeer_carry");
    {
        KTimer kt("k_qdeer_fixup_fwd", st);
#define FX(MPV) \
    hipLaunchKernelGGL((k_qdeer_fixup_fwd<MPV>), dim3(gridc), dim3(64), 0, st, coef, rhs, (const float *)carry, z, zalt, \
                       zsel, chain_bits, active, B, T, M, C, ncs)
        if (MP == 16) FX(16); else if (MP == 32) FX(32); else FX(64);
#undef FX
    }
    DEER_LAUNCH_CHECK("k_qdeer_fixup_fwd");
    return DEER_OK;
}

// chunks per block of the fused pass kernel (the chunk count per sequence is a multiple of it,
// at most QF_MAXG times it)
int qdeer_pass_group(int M) { return QF_WPB * (64 / q_padded(M)); }
int qdeer_pass_max_chunks(int M) { return QF_MAXG * qdeer_pass_group(M); }

int launch_qdeer_pass(const PlrnnArgs &a, float *z, float *zalt, const float *Pin, const float *vin, const double *gin,
                      float *Pout, float *vout, double *gout, int C, int ncs, const FusedCtl &fc, uint32_t *mark,
                      uint32_t pass_no, hipStream_t st) {
    const int MP = q_padded(a.M), GS = qdeer_pass_group(a.M);
    if (a.M < 1 || a.M > 64 || C < 1 || ncs < GS || ncs % GS || ncs > QF_MAXG * GS || (long)C * ncs < a.T ||
        (long)C * (ncs - GS) >= a.T ||
        !fc.seq || !fc.nd.pv || !Pin || !vin || !gin || !Pout || !vout || !gout)
    {
        set_error("fused quasi-DEER passes need M <= 64, a chunk count per sequence that is a multiple of %d, at "
                  "most %d, covering T with fewer than %d padding chunks, the control and two aggregate buffers",
                  GS, QF_MAXG * GS, GS);
        return DEER_ERR_INVALID_ARG;
    }
    KTimer kt("k_qdeer_pass", st);
    const unsigned grid = (unsigned)((long)a.B * ncs / GS);
#define QP(MPV)                                                                                                     \
    hipLaunchKernelGGL((k_qdeer_pass<MPV>), dim3(grid), dim3(64 * QF_WPB), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x, \
                       a.z0, z, zalt, a.T, a.M, C, ncs, Pin, vin, gin, Pout, vout, gout, fc, mark, pass_no, a.tw)
    if (MP == 16) QP(16); else if (MP == 32) QP(32); else QP(64);
#undef QP
    DEER_LAUNCH_CHECK("k_qdeer_pass");
    return DEER_OK;
}

int launch_qdeer_adjoint(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *coef, float *P,
                         float *v, float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st) {
    const int MP = q_padded(a.M);
    {
        KTimer kt("k_qdeer_resdiag", st);
        const dim3 grid = q_grid_rows(a.B, a.T, MP);
#define RD(MPV) \
    hipLaunchKernelGGL((k_qdeer_resdiag<MPV, true>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x, a.z0, z, \
                       z, (const int *)nullptr, (const int *)nullptr, (const float *)nullptr, (float *)nullptr, coef, \
                       a.B, a.T, a.M, a.tw)
        if (MP == 16) RD(16); else if (MP == 32) RD(32); else RD(64);
#undef RD
    }
    DEER_LAUNCH_CHECK("k_qdeer_resdiag<rev>");
    return launch_qdeer_scan_rev(a, g, seed_scale, z, coef, P, v, carry, lam, gpart, C, ncs, st);
}

int launch_qdeer_scan_rev(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, const float *coef,
                          float *P, float *v, float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st) {
    const int MP = q_padded(a.M);
    const int nchains = a.B * ncs;
    const int gridc = (nchains + 64 / MP - 1) / (64 / MP);
    {
        KTimer kt("k_qdeer_chunk", st);
#define CK(MPV) \
    hipLaunchKernelGGL((k_qdeer_chunk<MPV, true>), dim3(gridc), dim3(64), 0, st, coef, g, 1.f, z, a.x, \
                       seed_scale, a.N, (const int *)nullptr, P, v, a.B, a.T, a.M, C, ncs, a.tw)
        if (MP == 16) CK(16); else if (MP == 32) CK(32); else CK(64);
#undef CK
    }
    DEER_LAUNCH_CHECK("k_qdeer_chunk<rev>");
    {
        KTimer kt("k_qdeer_carry", st);
#define CR(MPV) \
    hipLaunchKernelGGL((k_qdeer_carry<MPV, true>), dim3(a.B), dim3(1024), 0, st, (const float *)P, (const float *)v, carry, \
                       (const int *)nullptr, a.M, ncs)
        if (MP == 16) CR(16); else if (MP == 32) CR(32); else CR(64);
#undef CR
    }
    DEER_LAUNCH_CHECK("k_qdeer_carry<rev>");
    {
        KTimer kt("k_qdeer_fixup_rev", st);
#define FX(MPV, GRV) \
    hipLaunchKernelGGL((k_qdeer_fixup_rev<MPV, GRV>), dim3(gridc), dim3(64), 0, st, coef, g, seed_scale, \
                       a.alpha, a.N, a.x, a.z0, z, (const float *)carry, lam, gpart, a.B, a.T, a.M, C, ncs, a.tw)
#define FXG(GRV) if (MP == 16) FX(16, GRV); else if (MP == 32) FX(32, GRV); else FX(64, GRV);
        if (gpart) { FXG(true) } else { FXG(false) }
#undef FXG
#undef FX
    }
    DEER_LAUNCH_CHECK("k_qdeer_fixup_rev");
    return DEER_OK;
}

}  // namespace deer
