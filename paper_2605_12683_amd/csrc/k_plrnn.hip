// Vanilla PLRNN path of GTF-DEER on gfx950:
//   z_t = diag(A) z~_{t-1} + W relu(z~_{t-1}) + h          (eq. shplrnn_nonlinear, V = I, b = 0)
//   J~_t = (diag(A) + W diag(m_t)) P_alpha                  (Jacobian of F, eq. error_forcing_decomp)
//
// Kernels (one Newton iteration = resjac -> chunk products -> carries -> fix-up):
//   k_resjac_plrnn     residual r_t, masks m_t (and optionally F, dense J~) at every step
//   k_chunk_product    per chunk of C steps: P_c = J~_e ... J~_s on the matrix cores (fp32
//                      MFMA) and v_c = the chunk's local solution from a zero carry (VALU)
//   k_carry            carries across chunks, one wave per sequence
//   k_fixup_fwd        Delta_t = J~_t Delta_{t-1} - r_t from the carry, z += Delta, max|Delta|
//   k_fixup_rev        lam_{t-1} = J~_t^T lam_t + g_{t-1} from the carry, fused parameter-
//                      gradient partial sums (gradients appendix)
//
// Padded dimension MP in {16, 32, 64} (the next one >= M); a wave holds NCH = 64/MP chains.
#include <type_traits>

#include "common.h"
#include "launch.h"
#include "newton_ctl.h"
#include "row16.h"

namespace deer {

template <int MP>
struct Geo {
    static constexpr int NCH = 64 / MP;   // chains (or timesteps) per wave
    static constexpr int NI = MP / 16;    // 16-row tiles
    static constexpr int NS = MP / 4;     // k-steps of the 16x16x4 MFMA
    static constexpr int MW = MP <= 32 ? 1 : 2;   // mask words per step
};

__device__ __forceinline__ float p_of(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

// Latent warm-up (section "Latent state warm-up", Alg. GTF-DEER): the forced inputs of steps
// s = 1..tw replace the observed latents by the data (alpha_s = 1, P_1), so those steps'
// Jacobians have the observed columns zeroed.  Kernels take it as a template flag WU; without it
// the warm-up code compiles away.  Step 0's Jacobian multiplies the fixed initial state's zero
// update, so it may count as a warm-up step too.
template <bool WU>
__device__ __forceinline__ float forced_in(float pi, float alpha, float zp, float xs, int s, int tw) {
    const float f = __fadd_rn(__fmul_rn(pi, zp), __fmul_rn(alpha, xs));
    if constexpr (WU) return s <= tw ? xs : f;
    return f;
}

__device__ __forceinline__ uint32_t mask_bit(const uint32_t *__restrict__ masks, size_t step, int MW, int i) {
    return (masks[step * MW + (i >> 5)] >> (i & 31)) & 1u;
}

// broadcast-read the MP values of chain n from LDS and dot them with row[] (registers)
template <int MP>
__device__ __forceinline__ float lds_dot(const float *lds, int n, const float *row) {
    const float4 *l4 = reinterpret_cast<const float4 *>(lds + n * MP);
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
    for (int q = 0; q < MP / 4; ++q) {
        float4 v = l4[q];
        acc0 = fmaf(row[4 * q + 0], v.x, acc0);
        acc1 = fmaf(row[4 * q + 1], v.y, acc1);
        acc0 = fmaf(row[4 * q + 2], v.z, acc0);
        acc1 = fmaf(row[4 * q + 3], v.w, acc1);
    }
    return acc0 + acc1;
}

// ---------------------------------------------------------------------------------------
// residual, masks, F and dense J~ at every (b, t)
// ---------------------------------------------------------------------------------------
template <int MP, bool DENSEJ>
__global__ __launch_bounds__(64) void k_resjac_plrnn(const float *__restrict__ A, const float *__restrict__ W,
                                                     const float *__restrict__ h, float alpha, int N,
                                                     const float *__restrict__ x, const float *__restrict__ z0,
                                                     const float *__restrict__ z, float *__restrict__ F_out,
                                                     float *__restrict__ r_out, float *__restrict__ J_out,
                                                     uint32_t *__restrict__ masks, const int *__restrict__ active,
                                                     int B, int T, int M) {
    using G = Geo<MP>;
    constexpr int NG = DENSEJ ? 1 : 4;    // groups of NCH rows handled per pass (memory parallelism)
    __shared__ __align__(16) float lds[NG][64];
    const int lane = threadIdx.x;
    const int n = lane / MP, i = lane % MP;
    float wrow[MP];
#pragma unroll
    for (int j = 0; j < MP; ++j) wrow[j] = (i < M && j < M) ? W[i * M + j] : 0.f;
    const float Ai = i < M ? A[i] : 0.f;
    const float hi = (h && i < M) ? h[i] : 0.f;
    const long total = (long)B * T;
    const long ngroups = (total + G::NCH - 1) / G::NCH;
    for (long grp0 = (long)blockIdx.x * NG; grp0 < ngroups; grp0 += (long)gridDim.x * NG) {
        float zt[NG], zc[NG];
        bool act[NG];
        long rowv[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const long row = (grp0 + q) * G::NCH + n;
            const bool in = row < total;
            const int b = in ? (int)(row / T) : 0, s = in ? (int)(row % T) : 0;
            act[q] = in && i < M && (!active || active[b]);
            rowv[q] = row;
            zt[q] = act[q] ? forced_state(x, z0, z, b, s, i, T, M, N, alpha) : 0.f;
            zc[q] = (act[q] && r_out) ? z[(size_t)row * M + i] : 0.f;
        }
        uint64_t bal[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const bool pos = zt[q] > 0.f;
            bal[q] = __ballot(pos);
            lds[q][lane] = pos ? zt[q] : 0.f;
        }
        lds_barrier();
        float F[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            F[q] = fmaf(Ai, zt[q], lds_dot<MP>(lds[q], n, wrow)) + hi;
            __builtin_amdgcn_sched_barrier(0);   // one dot product at a time: keeps the LDS reads of
                                                 // the other groups from being hoisted into registers
        }
        lds_barrier();
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const long row = rowv[q];
            if (act[q]) {
                const size_t e = (size_t)row * M + i;
                if (r_out) r_out[e] = zc[q] - F[q];
                if (F_out) F_out[e] = F[q];
                if (DENSEJ) {
                    float *Jr = J_out + ((size_t)row * M + i) * M;
#pragma unroll
                    for (int j = 0; j < MP; ++j) {
                        if (j < M) {
                            const float mj = (float)((bal[q] >> (n * MP + j)) & 1ull);
                            const float v = (j == i ? Ai : 0.f) + wrow[j] * mj;
                            Jr[j] = v * p_of(j, N, alpha);
                        }
                    }
                }
            }
            const bool in = row < total;
            if (masks && in && i == 0 && (!active || active[row / T])) {
                if (MP == 64) {
                    masks[(size_t)row * 2 + 0] = (uint32_t)bal[q];
                    if (M > 32) masks[(size_t)row * 2 + 1] = (uint32_t)(bal[q] >> 32);
                } else {
                    const uint64_t seg = bal[q] >> (n * MP);
                    masks[row] = (uint32_t)(MP == 32 ? seg : (seg & 0xffffull));
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// chunk aggregates.  Product over the step range [lo, hi) of the chain:
//   forward: P_c = J~_{s1-1} ... J~_{s0}           v_c = Delta_{s1-1} from a zero carry
//   reverse: P_c = J~_{s1} ... J~_{s0+1}  (then read transposed)
//            v_c = lam_{s0} of the chunk from lam_{s1} = 0
// MFMA formulation of P <- J~ P = diag(A p) P + (W diag(p)) (diag(m) P):
//   A operand = W diag(p) (constant, registers), B operand = the masked accumulator itself
//   (with the k-permutation kappa(4j+q, g) = 16j + 4g + q the 16x16x4 output layout is
//   exactly the B layout of the next step, so no data moves between steps).
// ---------------------------------------------------------------------------------------
template <int MP, bool REV, bool WU>
__global__ __launch_bounds__(64) void k_chunk_product_plrnn(
    const float *__restrict__ A, const float *__restrict__ W, float alpha, int N, const uint32_t *__restrict__ masks,
    const float *__restrict__ rhs, const float *__restrict__ z, const float *__restrict__ x, float seed_scale,
    float *__restrict__ Pout, float *__restrict__ vout, const int *__restrict__ active, int B, int T, int M, int C,
    int ncs, int tw) {
    using G = Geo<MP>;
    constexpr int NCH = G::NCH, NI = G::NI, NS = G::NS, MW = G::MW;
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

    // A operand: (W diag(p))[16I + c][16j + 4g + q]
    float Aop[NI][NS];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int j = 0; j < NS / 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int row = 16 * I + c, col = 16 * j + 4 * g + q;
                Aop[I][4 * j + q] = (row < M && col < M) ? W[row * M + col] * p_of(col, N, alpha) : 0.f;
            }
    float dI[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * I + 4 * g + r;
            dI[I][r] = row < M ? A[row] * p_of(row, N, alpha) : 0.f;
        }
    // latent warm-up steps (P_1): the observed latents' rows of the diagonal term are dropped
    float dIw[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) dIw[I][r] = (WU && 16 * I + 4 * g + r < N) ? 0.f : dI[I][r];
    // accumulators start at the identity of each chain
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

    // VALU chain for v_c: lane = (chain un, row ui)
    const int un = lane / MP, ui = lane % MP;
    float wv[MP];
    float du = 0.f, pu = 0.f, Au = 0.f;
    if (!REV) {
#pragma unroll
        for (int k = 0; k < MP; ++k) wv[k] = (ui < M && k < M) ? W[ui * M + k] * p_of(k, N, alpha) : 0.f;
        du = ui < M ? A[ui] * p_of(ui, N, alpha) : 0.f;
    } else {
#pragma unroll
        for (int k = 0; k < MP; ++k) wv[k] = (ui < M && k < M) ? W[k * M + ui] : 0.f;
        pu = p_of(ui, N, alpha);
        Au = ui < M ? A[ui] : 0.f;
    }
    int ub = 0, ulo = 0, uhi = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n)
        if (n == un) { ub = pb[n]; ulo = us0[n]; uhi = us1[n]; }
    float u = 0.f;

    for (int t = 0; t < maxlen; ++t) {
        // ---- matrix-core part: one step of every chain whose product is still running
#pragma unroll
        for (int Jt = 0; Jt < 4; ++Jt) {
            const int n = (16 * Jt) / MP;
            if (t < plen[n]) {
                const size_t step = (size_t)pb[n] * T + plo[n] + t;
                const uint32_t w0 = masks[step * MW];
                const uint32_t w1 = MW > 1 ? masks[step * MW + 1] : 0u;
                float Bop[NS];
#pragma unroll
                for (int j = 0; j < NS / 4; ++j) {
                    const uint32_t wj = (j >> 1) ? w1 : w0;
#pragma unroll
                    for (int q = 0; q < 4; ++q) Bop[4 * j + q] = select_bit(wj, 16 * (j & 1) + 4 * g + q, acc[j][Jt][q]);
                }
                const bool warm = WU && plo[n] + t <= tw;   // J~ of step plo + t with P_1
                if (warm) {
#pragma unroll
                    for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            if (16 * j + 4 * g + q < N) Bop[4 * j + q] = 0.f;
                }
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[I][Jt][r] *= warm ? dIw[I][r] : dI[I][r];
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int s = 0; s < NS; ++s) acc[I][Jt] = mfma16x16x4(Aop[I][s], Bop[s], acc[I][Jt]);
            }
        }
        // ---- VALU part: local solution of the chunk
        const bool run = ulo + t < uhi;
        if (!REV) {
            const int s = ulo + t;
            const size_t step = (size_t)ub * T + s;
            const float uo = (WU && ui < N && s <= tw) ? 0.f : u;   // P_s u
            float w = 0.f;
            if (run && ui < M) w = mask_bit(masks, step, MW, ui) ? uo : 0.f;
            lds[lane] = w;
            lds_barrier();
            const float y = fmaf(du, uo, lds_dot<MP>(lds, un, wv));
            lds_barrier();
            if (run && ui < M) u = y - rhs[step * M + ui];
        } else {
            const int k = uhi - 1 - t;    // lam_k = J~_{k+1}^T lam_{k+1} + g_k
            lds[lane] = u;
            lds_barrier();
            const float wt = lds_dot<MP>(lds, un, wv);
            lds_barrier();
            if (run && ui < M) {
                const size_t step = (size_t)ub * T + k;
                float y = 0.f;
                if (t > 0 && !(WU && ui < N && k + 1 <= tw)) {   // P_{k+1} = P_1 drops observed rows
                    const float m = (float)mask_bit(masks, step + 1, MW, ui);
                    y = pu * fmaf(Au, u, m * wt);
                }
                float gk;
                if (rhs) gk = rhs[step * M + ui];
                else gk = (ui < N && (!WU || k >= tw))
                              ? seed_scale * (z[step * M + ui] - x[((size_t)ub * (T + 1) + k + 1) * N + ui])
                              : 0.f;
                u = y + gk;
            }
        }
    }

    // ---- write the aggregates
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

// ---------------------------------------------------------------------------------------
// Forward Newton pass with the residual fused in: per step of every chain the wave forms
// z~_t, its ReLU ballot (which is at once the mask of the matrix-core bit select), F,
// r_t = z_t - F, and advances both the chunk product and the chunk-local solution.
// r and the masks are written for the fix-up pass.  Same MFMA layout as above.
// ---------------------------------------------------------------------------------------
template <int MP, bool WU>
__global__ __launch_bounds__(64) void k_newton_product_plrnn(
    const float *__restrict__ A, const float *__restrict__ W, const float *__restrict__ h, float alpha, int N,
    const float *__restrict__ x, const float *__restrict__ z0, const float *zbuf, const float *zalt,
    const int *__restrict__ zsel, float *__restrict__ r_out, uint32_t *__restrict__ masks, float *__restrict__ Pout,
    float *__restrict__ vout, const int *__restrict__ active, const float *__restrict__ gamma, int B, int T, int M, int C,
    int ncs, int tw) {
    using G = Geo<MP>;
    constexpr int NCH = G::NCH, NI = G::NI, NS = G::NS, MW = G::MW;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * NCH;
    int plen[NCH], cst[NCH];              // steps and first step of each chain
    float gam[NCH];                       // damping of the linearisation (1 = exact Newton)
    int maxlen = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n) {
        const int id = chain0 + n;
        bool ok = id < nchains;
        const int b = ok ? id / ncs : 0, cc = ok ? id % ncs : 0;
        ok = ok && (!active || active[b]);
        const int s0 = cc * C;
        plen[n] = ok ? min(C, T - s0) : 0;
        cst[n] = s0;
        gam[n] = gamma ? gamma[b] : 1.f;
        maxlen = max(maxlen, plen[n]);
    }
    float Aop[NI][NS];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int j = 0; j < NS / 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int row = 16 * I + c, col = 16 * j + 4 * g + q;
                Aop[I][4 * j + q] = (row < M && col < M) ? W[row * M + col] * p_of(col, N, alpha) : 0.f;
            }
    float dI[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * I + 4 * g + r;
            dI[I][r] = row < M ? A[row] * p_of(row, N, alpha) : 0.f;
        }
    if (NCH == 1) {   // one chain per wave: fold its damping into the operands once
#pragma unroll
        for (int I = 0; I < NI; ++I) {
#pragma unroll
            for (int s2 = 0; s2 < NS; ++s2) Aop[I][s2] *= gam[0];
#pragma unroll
            for (int r = 0; r < 4; ++r) dI[I][r] *= gam[0];
        }
    }
    // latent warm-up steps (P_1): the observed latents' rows of the diagonal term are dropped
    float dIw[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) dIw[I][r] = (WU && 16 * I + 4 * g + r < N) ? 0.f : dI[I][r];
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
    // lane-per-row part: lane = (chain un, latent ui)
    const int un = lane / MP, ui = lane % MP;
    const int uid = chain0 + un;
    const bool uok0 = uid < nchains;
    const int ub = uok0 ? uid / ncs : 0, us0 = uok0 ? (uid % ncs) * C : 0;
    int ulen = 0;
#pragma unroll
    for (int n = 0; n < NCH; ++n)
        if (n == un) ulen = plen[n];
    const bool lat = ui < M;
    float wrow[MP];
#pragma unroll
    for (int k = 0; k < MP; ++k) wrow[k] = (lat && k < M) ? W[ui * M + k] : 0.f;
    const float Ai = lat ? A[ui] : 0.f, hi = (lat && h) ? h[ui] : 0.f;
    const float pi = p_of(ui, N, alpha), di = Ai * pi;
    const bool forced = ui < N;
    float ugam = 1.f;
#pragma unroll
    for (int n = 0; n < NCH; ++n)
        if (n == un) ugam = gam[n];
    const float *z = cur_iter(zbuf, zalt, zsel, ub);   // this lane's sequence's iterate
    // z_{s-1} for the first step of the chunk
    float zprev = 0.f;
    if (ulen > 0 && lat) {
        if (us0 == 0) zprev = z0 ? z0[(size_t)ub * M + ui] : (forced ? x[(size_t)ub * (T + 1) * N + ui] : 0.f);
        else zprev = z[((size_t)ub * T + us0 - 1) * M + ui];
    }
    float u = 0.f;
    // z_s and x_s are loaded PD steps ahead (a queue shifted by one every step)
    constexpr int PD = 1;
    float zq[PD], xq[PD];
    auto fetch = [&](int t, float &zv, float &xv) {
        zv = 0.f;
        xv = 0.f;
        if (t < ulen && lat) {
            zv = z[((size_t)ub * T + us0 + t) * M + ui];
            if (forced) xv = x[((size_t)ub * (T + 1) + us0 + t) * N + ui];
        }
    };
#pragma unroll
    for (int q = 0; q < PD; ++q) fetch(q, zq[q], xq[q]);
    for (int t = 0; t < maxlen; ++t) {
        const bool run = t < ulen && lat;
        const int s = us0 + t;
        const float zcur = zq[0], xb = xq[0];
#pragma unroll
        for (int q = 0; q + 1 < PD; ++q) {
            zq[q] = zq[q + 1];
            xq[q] = xq[q + 1];
        }
        fetch(t + PD, zq[PD - 1], xq[PD - 1]);
        // forced state of this step (s == 0: z_0 itself)
        float zt = 0.f;
        if (run) {
            if (s == 0 || !forced) zt = zprev;
            else zt = forced_in<WU>(pi, alpha, zprev, xb, s, tw);
        }
        const bool pos = zt > 0.f;
        const uint64_t bal = __ballot(pos);
        lds[lane] = pos ? zt : 0.f;
        lds_barrier();
        const float F = fmaf(Ai, zt, lds_dot<MP>(lds, un, wrow)) + hi;
        lds_barrier();
        const float r = zcur - F;
        if (run) {
            const size_t e = ((size_t)ub * T + s) * M + ui;
            r_out[e] = r;
            if (ui == 0) {
                const size_t step = (size_t)ub * T + s;
                if (MP == 64) {
                    masks[step * 2] = (uint32_t)bal;
                    if (M > 32) masks[step * 2 + 1] = (uint32_t)(bal >> 32);
                } else {
                    const uint64_t seg = bal >> (un * MP);
                    masks[step] = (uint32_t)(MP == 32 ? seg : (seg & 0xffffull));
                }
            }
        }
        // matrix-core step of every chain still running
#pragma unroll
        for (int Jt = 0; Jt < 4; ++Jt) {
            const int n = (16 * Jt) / MP;
            if (t < plen[n]) {
                const uint64_t seg = bal >> (n * MP);
                const uint32_t w0 = (uint32_t)seg;
                const uint32_t w1 = (uint32_t)(seg >> 32);
                float Bop[NS];
#pragma unroll
                for (int j = 0; j < NS / 4; ++j) {
                    const uint32_t wj = (j >> 1) ? w1 : w0;
#pragma unroll
                    for (int q = 0; q < 4; ++q) Bop[4 * j + q] = select_bit(wj, 16 * (j & 1) + 4 * g + q, acc[j][Jt][q]);
                }
                const bool warm = WU && cst[n] + t <= tw;   // P_1: the observed latents' rows dropped
                if (warm) {
#pragma unroll
                    for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            if (16 * j + 4 * g + q < N) Bop[4 * j + q] = 0.f;
                }
                if (NCH > 1 && gam[n] != 1.f) {   // damped chain (uniform branch)
                    const float gm = gam[n];
#pragma unroll
                    for (int s2 = 0; s2 < NS; ++s2) Bop[s2] *= gm;
#pragma unroll
                    for (int I = 0; I < NI; ++I)
#pragma unroll
                        for (int r2 = 0; r2 < 4; ++r2) acc[I][Jt][r2] *= gm;
                }
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2) acc[I][Jt][r2] *= warm ? dIw[I][r2] : dI[I][r2];
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int s2 = 0; s2 < NS; ++s2) acc[I][Jt] = mfma16x16x4(Aop[I][s2], Bop[s2], acc[I][Jt]);
            }
        }
        // chunk-local solution: u <- gamma (d u + W (p m u)) - r
        const float uo = (WU && forced && us0 + t <= tw) ? 0.f : u;   // P_s u
        lds[lane] = pos ? pi * uo : 0.f;
        lds_barrier();
        const float y = fmaf(di, uo, lds_dot<MP>(lds, un, wrow));
        lds_barrier();
        if (run) {
            u = fmaf(ugam, y, -r);
            zprev = zcur;
        }
    }
#pragma unroll
    for (int Jt = 0; Jt < 4; ++Jt) {
        const int n = (16 * Jt) / MP;
        const int id = chain0 + n;
        if (id < nchains && plen[n] > 0) {
            const int col = 16 * Jt + c - n * MP;
            float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) P[(16 * I + 4 * g + r2) * MP + col] = acc[I][Jt][r2];
        }
    }
    if (uok0) vout[(size_t)uid * MP + ui] = u;
}

// A-operand fragments of a 16 x 16 map (P_c, or its transpose) and the vector v_c for the
// matrix-core carries: lane (g, c) takes row c, columns 4g..4g+3 (transposed: rows 4g..4g+3 of
// column c) and v_c[4g..4g+3]
template <bool REV>
__device__ __forceinline__ void carry16_fetch(const float *__restrict__ Pc, const float *__restrict__ vc, int g, int c,
                                              float (&a)[4], float (&vv)[4]) {
    if (!REV) {
        const float4 t = *reinterpret_cast<const float4 *>(Pc + c * 16 + 4 * g);
        a[0] = t.x; a[1] = t.y; a[2] = t.z; a[3] = t.w;
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) a[q] = Pc[(4 * g + q) * 16 + c];
    }
    const float4 u = *reinterpret_cast<const float4 *>(vc + 4 * g);
    vv[0] = u.x; vv[1] = u.y; vv[2] = u.z; vv[3] = u.w;
}

// ---------------------------------------------------------------------------------------
// M <= 16: register-tiled forward Newton pass and fix-up.
// A wave holds four chains, one per 16-lane row (lane = 16 * chain + latent), so a row of the
// wave is one chain's state vector and the products W y of F and of the chunk-local solution
// are formed with DPP row rotations (no LDS, no barrier).  Steps go in tiles of TB.  In a tile
// that all four chains run to its end (every tile but a ragged chunk's last) all loads of the
// tile are issued at once through buffer resources (one lane offset for all of them), the
// residual of every step of the tile, which does not depend on the recurrence, is formed
// first, and the serial part then runs from registers, with the matrix-core updates of the
// four chains free of branches so that they interleave.  Other tiles go step by step.  The
// residual and the masks stay in registers: the fix-up forms them again from z and x.
// ---------------------------------------------------------------------------------------


__device__ __forceinline__ int rfl_i(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float rfl_f(float v) { return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v))); }

// the wave's four chains: sequence and chunk index, lengths, damping, and whether they all read
// one iterate buffer.  chain0 is wave-uniform, so every value here is scalar; the control words
// of the four chains are loaded at once (clamped indices) and combined afterwards.
struct Chains16 {
    int plen[4];
    int cs[4];   // first step of each chain in its sequence
    float gam[4];
    int minlen, maxlen;
    bool onebuf;
};
__device__ __forceinline__ Chains16 chains16(int chain0, int nchains, int ncs, int C, int T,
                                             const int *__restrict__ active, const float *__restrict__ gamma,
                                             const int *__restrict__ zsel) {
    Chains16 w;
    const int b0 = chain0 / ncs, c0 = chain0 - b0 * ncs;
    int act[4], sel[4], bq[4], cq[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        int bb = b0, cc = c0 + n;
#pragma unroll
        for (int k = 0; k < 3; ++k)   // c0 + n < c0 + 4 <= 4 ncs
            if (cc >= ncs) {
                cc -= ncs;
                ++bb;
            }
        const bool ok = chain0 + n < nchains;
        bq[n] = ok ? bb : 0;
        cq[n] = ok ? cc : 0;
        act[n] = active ? active[bq[n]] : 1;
        w.gam[n] = gamma ? gamma[bq[n]] : 1.f;
        sel[n] = zsel ? zsel[bq[n]] : 0;
    }
    w.minlen = C;
    w.maxlen = 0;
    w.onebuf = true;
    int sel0 = -1;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const bool ok = chain0 + n < nchains && act[n] != 0;
        w.plen[n] = ok ? min(C, T - cq[n] * C) : 0;
        w.cs[n] = cq[n] * C;
        if (w.plen[n] > 0) {
            if (sel0 >= 0 && sel[n] != sel0) w.onebuf = false;
            sel0 = sel[n];
        }
        w.minlen = min(w.minlen, w.plen[n]);
        w.maxlen = max(w.maxlen, w.plen[n]);
    }
    return w;
}

// sequence b and first step s0 of chain chain0 + g (g < 4) without a division (chain0 is
// uniform); 0, 0 past the last chain
__device__ __forceinline__ void chain_pos(int chain0, int g, int nchains, int ncs, int C, int &b, int &s0) {
    const int b0 = chain0 / ncs;
    int bb = b0, cc = chain0 - b0 * ncs + g;
#pragma unroll
    for (int k = 0; k < 3; ++k)
        if (cc >= ncs) {
            cc -= ncs;
            ++bb;
        }
    const bool ok = chain0 + g < nchains;
    b = ok ? bb : 0;
    s0 = ok ? cc * C : 0;
}

// acc[n] *= gamma_n^(steps chain n ran in the tile [t0, t0 + tl)): J~ = gamma (...) per step
__device__ __forceinline__ void damp_tile(v4f (&acc)[4], const Chains16 &w, int t0, int tl) {
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const float gm = w.gam[n];
        if (gm != 1.f) {
            const int steps = max(0, min(tl, w.plen[n] - t0));
            float gp = 1.f;
            for (int k = 0; k < steps; ++k) gp *= gm;
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) acc[n][r2] *= gp;
        }
    }
}

// one matrix-core step of chain n: acc <- (diag(d) + W p diag(m)) acc.  The mask and the
// diagonal go into the A operand: lane (g, c) supplies, for k = 4 g + q, m_k ? WpD[q] : Dq[q]
// with WpD = (W p)[c][k] + [c == k] d_k and Dq = [c == k] d_k, so B is the product unchanged.
__device__ __forceinline__ v4f mfma_step16(const v4f &acc, uint32_t wn, int g, const float (&WpD)[4],
                                           const float (&Dq)[4]) {
    v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)wn, 4 * g + q, 1);
        const float a = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
        nx = mfma16x16x4(a, acc[q], nx);
    }
    return nx;
}

// bits tt < n of a tile's step mask (n may lie outside 0..32)
__device__ __forceinline__ uint32_t low_bits(int n) { return n <= 0 ? 0u : (n >= 32 ? ~0u : (1u << n) - 1u); }

// forced input of an observed latent at tile row tt; in a tile holding warm-up steps, bit tt of
// wb marks one (the data itself, alpha_s = 1)
template <bool WT>
__device__ __forceinline__ float forced_at(float pi, float alpha, float zp, float xs, uint32_t wb, int tt) {
    const float f = __fadd_rn(__fmul_rn(pi, zp), __fmul_rn(alpha, xs));
    if constexpr (WT) return ((wb >> tt) & 1u) ? xs : f;
    return f;
}

// mfma_step16 in a warm-up step: the product's rows of the observed latents (fr[q]: row
// 4 g + q) are left out of the B operand, which is J~ = J_F P_1 acting on it
__device__ __forceinline__ v4f mfma_step16_warm(const v4f &acc, uint32_t wn, int g, const float (&WpD)[4],
                                                const float (&Dq)[4], const bool (&fr)[4]) {
    v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)wn, 4 * g + q, 1);
        const float a = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
        nx = mfma16x16x4(a, fr[q] ? 0.f : acc[q], nx);
    }
    return nx;
}

// WPB waves per block (1, or 8 for the group maps: the block's 32 chunks then belong to one
// sequence); wmaps: 0 plain chunk aggregates, 1 wave maps, 2 wave maps composed per block into
// group maps (gmap).
template <int TB, int WPB, bool WU>
__global__ __launch_bounds__(64 * WPB) void k_newton_product_plrnn16(
    const float *__restrict__ A, const float *__restrict__ W, const float *__restrict__ h, float alpha, int N,
    const float *__restrict__ x, const float *__restrict__ z0, const float *zbuf, const float *zalt,
    const int *__restrict__ zsel, float *__restrict__ Pout,
    float *__restrict__ vout, const int *__restrict__ active, const float *__restrict__ gamma, int B, int T, int M, int C,
    int ncs, int wmaps, float *__restrict__ gmap, uint32_t *mark, uint32_t pass_no, int tw) {
    // the wave index is uniform: the chain set, its control words and the tile addresses are
    // scalar values (scalar loads, no per-lane address arithmetic)
    const int lane = threadIdx.x & 63, wvb = WPB > 1 ? rfl_i((int)(threadIdx.x >> 6)) : 0, g = lane >> 4, c = lane & 15;
    if (mark && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(mark, pass_no, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const int nchains = B * ncs;
    const int chain0 = (blockIdx.x * WPB + wvb) * 4;
    const Chains16 w = chains16(chain0, nchains, ncs, C, T, active, gamma, zsel);
    if (w.maxlen == 0) return;
    // row part: this lane is latent c of chain g
    const int id = chain0 + g;
    const bool okc = id < nchains;
    int b, s0;
    chain_pos(chain0, g, nchains, ncs, C, b, s0);
    int len = 0;
    float ugam = 1.f;
#pragma unroll
    for (int n = 0; n < 4; ++n)
        if (n == g) {
            len = w.plen[n];
            ugam = w.gam[n];
        }
    const bool lat = c < M, forced = c < N;
    bool fr[4];   // B-operand rows 4 g + q of observed latents (dropped in warm-up steps)
#pragma unroll
    for (int q = 0; q < 4; ++q) fr[q] = 4 * g + q < N;
    // tile resources, based at the first row of the wave's first chain
    const int b0 = chain0 / ncs, s00 = (chain0 % ncs) * C;
    const size_t row0 = (size_t)b0 * T + s00, xrow0 = (size_t)b0 * (T + 1) + s00;
    const uint32_t drow = (uint32_t)((size_t)b * T + s0 - row0), dxrow = (uint32_t)((size_t)b * (T + 1) + s0 - xrow0);
    const float *zw = cur_iter(zbuf, zalt, zsel, b0);
    const auto rz = wave_rsrc(zw + row0 * M);
    const auto rx = wave_rsrc(N > 0 ? x + xrow0 * N : zw);
    const uint32_t vz = lat ? 4u * (drow * M + c) : kOffLane;
    const uint32_t vx = forced ? 4u * (dxrow * N + c) : kOffLane;
    // the first tile's loads go out before the weights are gathered
    float zv[TB], xv[TB];
    if (w.onebuf && TB <= w.minlen) {
#pragma unroll
        for (int tt = 0; tt < TB; ++tt) {
            zv[tt] = bload(rz, vz, 4 * tt * M);
            xv[tt] = bload(rx, vx, 4 * tt * N);
        }
    }
    const float *z = cur_iter(zbuf, zalt, zsel, b);
    float zprev = 0.f;
    if (len > 0 && lat) {
        if (s0 == 0) zprev = z0 ? z0[(size_t)b * M + c] : (forced ? x[(size_t)b * (T + 1) * N + c] : 0.f);
        else zprev = z[((size_t)b * T + s0 - 1) * M + c];
    }
    float WpD[4], Dq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int col = 4 * g + q;
        const float wp = (c < M && col < M) ? W[c * M + col] * p_of(col, N, alpha) : 0.f;
        Dq[q] = (col == c && col < M) ? A[col] * p_of(col, N, alpha) : 0.f;
        WpD[q] = wp + Dq[q];
    }
    v4f acc[4];
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[n][r] = (4 * g + r == c) ? 1.f : 0.f;
    int src[16];
    row_sources(c, src);
    float wr[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) wr[k] = (lat && src[k] < M) ? W[c * M + src[k]] : 0.f;
    const float Ai = lat ? A[c] : 0.f, hi = (lat && h) ? h[c] : 0.f;
    const float pi = p_of(c, N, alpha), di = Ai * pi;
    float u = 0.f;
    for (int t0 = 0; t0 < w.maxlen; t0 += TB) {
        const int tl = min(TB, w.maxlen - t0);
        if (w.onebuf && t0 + TB <= w.minlen) {
            if (t0 > 0) {
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    zv[tt] = bload(rz, vz, 4 * (t0 + tt) * M);
                    xv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);
                }
            }
            bool wtile = false;   // some chain of the wave has a latent warm-up step in this tile
            if constexpr (WU) {
#pragma unroll
                for (int n = 0; n < 4; ++n) wtile = wtile || w.cs[n] + t0 <= tw;
            }
            if (wtile) {
                // the tile body below with the warm-up steps' P_1: the observed latents' rows of
                // the B operand and of u dropped, their forced inputs the data
                const uint32_t wb = low_bits(tw - (s0 + t0) + 1);   // bit tt: s0 + t0 + tt <= tw
                int lim[4];   // chain n: tile steps tt < lim[n] are warm-up steps
#pragma unroll
                for (int n = 0; n < 4; ++n) lim[n] = tw - (w.cs[n] + t0) + 1;
                uint32_t posb = 0u;
#pragma unroll
                for (int tt = 0; tt < TB; tt += 2) {
                    const int s = s0 + t0 + tt;
                    const float zt0 = (s == 0 || !forced) ? zprev : forced_at<true>(pi, alpha, zprev, xv[tt], wb, tt);
                    const float zt1 = !forced ? zv[tt] : forced_at<true>(pi, alpha, zv[tt], xv[tt + 1], wb, tt + 1);
                    const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                    posb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                    float d0, d1;
                    row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                    const float F0 = fmaf(Ai, zt0, d0) + hi, F1 = fmaf(Ai, zt1, d1) + hi;
                    zprev = zv[tt + 1];
                    zv[tt] = zv[tt] - F0;
                    zv[tt + 1] = zv[tt + 1] - F1;
                }
                const uint32_t wf = forced ? wb : 0u;
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool pos = (posb >> tt) & 1u;
                    const uint64_t bal = __ballot(pos);
                    float Am[4][4];
#pragma unroll
                    for (int n = 0; n < 4; ++n)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t m =
                                (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                            Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                        }
                    v4f nx[4];
#pragma unroll
                    for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int q = 0; q < 4; ++q)
#pragma unroll
                        for (int n = 0; n < 4; ++n)
                            nx[n] = mfma16x16x4(Am[n][q], (fr[q] && tt < lim[n]) ? 0.f : acc[n][q], nx[n]);
#pragma unroll
                    for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                    const float uo = ((wf >> tt) & 1u) ? 0.f : u;
                    const float y = fmaf(di, uo, row16_dot(wr, pos ? pi * uo : 0.f));
                    u = fmaf(ugam, y, -zv[tt]);
                }
            } else {
                // residual and masks of every step of the tile, two steps at a time; r overwrites zv
                uint32_t posb = 0u;
#pragma unroll
                for (int tt = 0; tt < TB; tt += 2) {
                    const int s = s0 + t0 + tt;
                    const float zt0 =
                        (s == 0 || !forced) ? zprev : __fadd_rn(__fmul_rn(pi, zprev), __fmul_rn(alpha, xv[tt]));
                    const float zt1 =
                        !forced ? zv[tt] : __fadd_rn(__fmul_rn(pi, zv[tt]), __fmul_rn(alpha, xv[tt + 1]));
                    const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                    posb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                    float d0, d1;
                    row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                    const float F0 = fmaf(Ai, zt0, d0) + hi, F1 = fmaf(Ai, zt1, d1) + hi;
                    zprev = zv[tt + 1];
                    zv[tt] = zv[tt] - F0;
                    zv[tt + 1] = zv[tt + 1] - F1;
                }
                // serial part: chunk products and chunk-local solutions
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool pos = (posb >> tt) & 1u;
                    const uint64_t bal = __ballot(pos);
                    // the four chains' updates interleaved: k-slice outer, chain inner
                    float Am[4][4];
#pragma unroll
                    for (int n = 0; n < 4; ++n)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t m =
                                (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                            Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                        }
                    v4f nx[4];
#pragma unroll
                    for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int q = 0; q < 4; ++q)
#pragma unroll
                        for (int n = 0; n < 4; ++n) nx[n] = mfma16x16x4(Am[n][q], acc[n][q], nx[n]);
#pragma unroll
                    for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                    const float y = fmaf(di, u, row16_dot(wr, pos ? pi * u : 0.f));
                    u = fmaf(ugam, y, -zv[tt]);
                }
            }
        } else {
            for (int t = t0; t < t0 + tl; ++t) {
                const bool run = t < len && lat;
                const int s = s0 + t;
                float zcur = 0.f, xb = 0.f;
                if (run) {
                    zcur = z[((size_t)b * T + s) * M + c];
                    if (forced && s > 0) xb = x[((size_t)b * (T + 1) + s) * N + c];
                }
                float zt = 0.f;
                if (run) zt = (s == 0 || !forced) ? zprev : forced_in<WU>(pi, alpha, zprev, xb, s, tw);
                const bool pos = zt > 0.f;
                const uint64_t bal = __ballot(pos);
                const float F = fmaf(Ai, zt, row16_dot(wr, pos ? zt : 0.f)) + hi;
                const float r = zcur - F;
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    if (t < w.plen[n]) {
                        if (WU && w.cs[n] + t <= tw)
                            acc[n] = mfma_step16_warm(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq, fr);
                        else
                            acc[n] = mfma_step16(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq);
                    }
                float uo = u;
                if constexpr (WU) uo = (forced && s <= tw) ? 0.f : u;
                const float y = fmaf(di, uo, row16_dot(wr, pos ? pi * uo : 0.f));
                if (run) {
                    u = fmaf(ugam, y, -r);
                    zprev = zcur;
                }
            }
        }
        damp_tile(acc, w, t0, tl);
    }
    if (wmaps) {
        // The wave's four chunks (one sequence, all active) composed for the carry pass:
        //   slot chain0:      wave map  Q = P_3 P_2 P_1 P_0,  u_w = the four chunks' walk from 0
        //   slot chain0 + n:  prefix    R_n = P_{n-1} ... P_0, s_n = the walk of the first n chunks
        // so that carry(chain0 + n) = R_n carry(chain0) + s_n.  A chunk product in accumulator
        // layout is transposed through LDS into the A-operand layout; vectors ride in column 0.
        __shared__ float lt[WPB][3][16][17];
        __shared__ float lv[WPB][4][16];
#pragma unroll
        for (int n = 1; n < 4; ++n)
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) lt[wvb][n - 1][4 * g + r2][c] = acc[n][r2];
        lv[wvb][g][c] = u;
        wave_lds_sync();   // each wave's own slots
        float Am[3][4];
        v4f bv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int n = 1; n < 4; ++n) Am[n - 1][q] = lt[wvb][n - 1][c][4 * g + q];
#pragma unroll
            for (int n = 0; n < 4; ++n) bv[n][q] = c == 0 ? lv[wvb][n][4 * g + q] : 0.f;
        }
        v4f R2 = {0.f, 0.f, 0.f, 0.f}, R3 = {0.f, 0.f, 0.f, 0.f}, Qw = {0.f, 0.f, 0.f, 0.f};
        v4f s2 = bv[1], s3 = bv[2], uw = bv[3];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            R2 = mfma16x16x4(Am[0][q], acc[0][q], R2);
            s2 = mfma16x16x4(Am[0][q], bv[0][q], s2);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            R3 = mfma16x16x4(Am[1][q], R2[q], R3);
            s3 = mfma16x16x4(Am[1][q], s2[q], s3);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            Qw = mfma16x16x4(Am[2][q], R3[q], Qw);
            uw = mfma16x16x4(Am[2][q], s3[q], uw);
        }
        const v4f outm[4] = {Qw, acc[0], R2, R3}, outv[4] = {uw, bv[0], s2, s3};
#pragma unroll
        for (int n = (WPB > 1 ? 1 : 0); n < 4; ++n) {
            float *P = Pout + (size_t)(chain0 + n) * 256;
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = outm[n][r2];
            if (c == 0)
                *reinterpret_cast<float4 *>(vout + (size_t)(chain0 + n) * 16 + 4 * g) =
                    make_float4(outv[n][0], outv[n][1], outv[n][2], outv[n][3]);
        }
        if (WPB > 1) {
            // group maps: wave 0 composes the block's eight wave maps in order; slot chain0 of
            // wave k receives the composition of waves 0..k-1 (carry(wave k) = G_k carry(group)
            // + g_k), and gmap[b][group] the whole group's map
            __shared__ float lq[WPB][16][17];
            __shared__ float lu[WPB][16];
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) lq[wvb][4 * g + r2][c] = Qw[r2];
            if (c == 0) {
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) lu[wvb][4 * g + r2] = uw[r2];
            }
            __syncthreads();
            if (wvb != 0) return;
            const int bc0 = blockIdx.x * WPB * 4;   // the block's first chain
            v4f Gm, gu = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) Gm[r2] = (4 * g + r2 == c) ? 1.f : 0.f;
            for (int k = 0; k < WPB; ++k) {
                float *P = Pout + (size_t)(bc0 + 4 * k) * 256;
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = Gm[r2];
                if (c == 0)
                    *reinterpret_cast<float4 *>(vout + (size_t)(bc0 + 4 * k) * 16 + 4 * g) =
                        make_float4(gu[0], gu[1], gu[2], gu[3]);
                v4f ng = {0.f, 0.f, 0.f, 0.f}, nu;
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) nu[r2] = c == 0 ? lu[k][4 * g + r2] : 0.f;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float aq = lq[k][c][4 * g + q];
                    ng = mfma16x16x4(aq, Gm[q], ng);
                    nu = mfma16x16x4(aq, gu[q], nu);
                }
                Gm = ng;
                gu = nu;
            }
            const int ngm = ncs / (4 * WPB);
            float *Gp = gmap + ((size_t)(bc0 / ncs) * ngm + (bc0 % ncs) / (4 * WPB)) * 272;
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) Gp[(4 * g + r2) * 16 + c] = Gm[r2];
            if (c == 0) *reinterpret_cast<float4 *>(Gp + 256 + 4 * g) = make_float4(gu[0], gu[1], gu[2], gu[3]);
        }
        return;
    }
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const int cid = chain0 + n;
        if (cid < nchains && w.plen[n] > 0) {
            float *P = Pout + (size_t)cid * 256;
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = acc[n][r2];
        }
    }
    if (okc) vout[(size_t)id * 16 + c] = u;
}

// M <= 16 forward fix-up.  The residual and the masks are formed again here from z and x (the
// same operations as the forward pass, so the same values), which saves writing them there
// and reading them here; Delta_t = gamma (diag(d) + W p diag(m_t)) Delta_{t-1} - r_t from the
// chunk's carry, z + Delta written to the other iterate buffer, per-chain max |Delta| and max
// |z|, and (with fc.seq) the pass-end control of the sequence.
template <int TB, bool WU>
__global__ __launch_bounds__(64) void k_fixup_fwd_plrnn16(const float *__restrict__ A, const float *__restrict__ W,
                                                          const float *__restrict__ h, float alpha, int N,
                                                          const float *__restrict__ x, const float *__restrict__ z0,
                                                          const float *__restrict__ carry_in, float *zbuf,
                                                          float *zalt, const int *__restrict__ zsel,
                                                          uint32_t *__restrict__ chain_bits,
                                                          const int *__restrict__ active,
                                                          const float *__restrict__ gamma, int B, int T, int M, int C,
                                                          int ncs, const float *__restrict__ Pm,
                                                          const float *__restrict__ vmap,
                                                          const float *__restrict__ gmap, FusedCtl fc, int tw) {
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * 4;
    const Chains16 w = chains16(chain0, nchains, ncs, C, T, active, gamma, zsel);
    if (w.maxlen == 0) return;
    const int id = chain0 + g;
    const bool okc = id < nchains;
    int b, s0;
    chain_pos(chain0, g, nchains, ncs, C, b, s0);
    int len = 0;
    float gm = 1.f;
#pragma unroll
    for (int n = 0; n < 4; ++n)
        if (n == g) {
            len = w.plen[n];
            gm = w.gam[n];
        }
    const bool lat = c < M, forced = c < N;
    int src[16];
    row_sources(c, src);
    float wr[16], wp[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        wr[k] = (lat && src[k] < M) ? W[c * M + src[k]] : 0.f;
        wp[k] = wr[k] * p_of(src[k], N, alpha);
    }
    const float Ai = lat ? A[c] : 0.f, hi = (lat && h) ? h[c] : 0.f;
    const float pi = p_of(c, N, alpha), d = Ai * pi;
    float D = 0.f;
    // group maps: the wave's carry is walked here from the sequence start over the group maps
    // before the wave's group (four MFMAs a step, maps eight steps ahead), then taken through
    // the wave's prefix in its group (slot chain0)
    __shared__ float wcs[16];
    if (gmap) {
        const int ngm = ncs / 32, grp = (chain0 % ncs) / 32, bq = chain0 / ncs;
        const float *Gb = gmap + (size_t)bq * ngm * 272;
        v4f cur = {0.f, 0.f, 0.f, 0.f};
        constexpr int PF = 8;
        float ga[PF][4], gv[PF][4];
        if (grp > 0) {
#pragma unroll
            for (int d2 = 0; d2 < PF; ++d2) {
                const float *Gk = Gb + (size_t)min(d2, grp - 1) * 272;
                carry16_fetch<false>(Gk, Gk + 256, g, c, ga[d2], gv[d2]);
            }
        }
        for (int k0 = 0; k0 < grp; k0 += PF) {
#pragma unroll
            for (int d2 = 0; d2 < PF; ++d2) {
                if (k0 + d2 >= grp) break;
                v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) nx = mfma16x16x4(ga[d2][q], cur[q], nx);
                if (c == 0) {
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2) nx[r2] += gv[d2][r2];
                }
                cur = nx;
                const float *Gk = Gb + (size_t)min(k0 + d2 + PF, grp - 1) * 272;
                carry16_fetch<false>(Gk, Gk + 256, g, c, ga[d2], gv[d2]);
            }
        }
        {
            float wa[4], wvv[4];
            carry16_fetch<false>(Pm + (size_t)chain0 * 256, vmap + (size_t)chain0 * 16, g, c, wa, wvv);
            v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) nx = mfma16x16x4(wa[q], cur[q], nx);
            if (c == 0) {
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) wcs[4 * g + r2] = nx[r2] + wvv[r2];
            }
        }
        lds_barrier();
    }
    if (len > 0 && lat) {
        if (!Pm || (g == 0 && !gmap)) {
            D = carry_in[(size_t)id * 16 + c];
        } else if (g == 0) {
            D = wcs[c];
        } else {   // composed wave maps: carry = R_g carry(chain0) + s_g
            const float4 *R4 = reinterpret_cast<const float4 *>(Pm + (size_t)id * 256 + c * 16);
            const float4 *w4 = gmap ? reinterpret_cast<const float4 *>(wcs)
                                    : reinterpret_cast<const float4 *>(carry_in + (size_t)chain0 * 16);
            float a0 = vmap[(size_t)id * 16 + c], a1 = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 rr4 = R4[q], ww = w4[q];
                a0 = fmaf(rr4.x, ww.x, a0);
                a1 = fmaf(rr4.y, ww.y, a1);
                a0 = fmaf(rr4.z, ww.z, a0);
                a1 = fmaf(rr4.w, ww.w, a1);
            }
            D = a0 + a1;
        }
    }
    const float *zin = cur_iter(zbuf, zalt, zsel, b);
    float *zout = next_iter(zbuf, zalt, zsel, b);
    float zprev = 0.f;   // z_{s-1} of the first step (the initial state at s = 0)
    if (len > 0 && lat) {
        if (s0 == 0) zprev = z0 ? z0[(size_t)b * M + c] : (forced ? x[(size_t)b * (T + 1) * N + c] : 0.f);
        else zprev = zin[((size_t)b * T + s0 - 1) * M + c];
    }
    const int cl0 = min(chain0, nchains - 1);   // a wave past the last chain touches no memory
    const int b0 = cl0 / ncs, s00 = (cl0 % ncs) * C;
    const size_t row0 = (size_t)b0 * T + s00, xrow0 = (size_t)b0 * (T + 1) + s00;
    const uint32_t drow = (uint32_t)((size_t)b * T + s0 - row0);
    const uint32_t dxrow = (uint32_t)((size_t)b * (T + 1) + s0 - xrow0);
    const auto rzi = wave_rsrc(cur_iter(zbuf, zalt, zsel, b0) + row0 * M);
    const auto rzo = wave_rsrc(next_iter(zbuf, zalt, zsel, b0) + row0 * M);
    const auto rx = wave_rsrc(N > 0 ? x + xrow0 * N : zin);
    const uint32_t vz = lat ? 4u * (drow * M + c) : kOffLane;
    const uint32_t vx = forced ? 4u * (dxrow * N + c) : kOffLane;
    uint32_t emax = 0u, zmax = 0u;
    for (int t0 = 0; t0 < w.maxlen; t0 += TB) {
        const int tl = min(TB, w.maxlen - t0);
        if (w.onebuf && t0 + TB <= w.minlen) {
            float zv[TB], rv[TB];
#pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                zv[tt] = bload(rzi, vz, 4 * (t0 + tt) * M);
                rv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);   // x of the step, replaced by r below
            }
            // a tile holding latent warm-up steps of this lane's chunk runs the body with P_1 there
            bool wtile = false;
            if constexpr (WU) {
#pragma unroll
                for (int n = 0; n < 4; ++n) wtile = wtile || w.cs[n] + t0 <= tw;
            }
            if (wtile) {
                const uint32_t wb = low_bits(tw - (s0 + t0) + 1);   // bit tt: s0 + t0 + tt <= tw
                const uint32_t wf = forced ? wb : 0u;
                // residual and masks of the tile (as in the forward pass)
                uint32_t mb = 0u;
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const int s = s0 + t0 + tt;
                    const float zt = (s == 0 || !forced) ? zprev : forced_at<true>(pi, alpha, zprev, rv[tt], wb, tt);
                    const bool pos = zt > 0.f;
                    mb |= (pos ? 1u : 0u) << tt;
                    const float F = fmaf(Ai, zt, row16_dot(wr, pos ? zt : 0.f)) + hi;
                    zprev = zv[tt];
                    rv[tt] = zv[tt] - F;
                }
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool m = (mb >> tt) & 1u;
                    const float Do = ((wf >> tt) & 1u) ? 0.f : D;   // P_1: observed entries dropped
                    const float y = fmaf(d, Do, row16_dot(wp, m ? Do : 0.f));
                    D = fmaf(gm, y, -rv[tt]);
                    const float zc = zv[tt];
                    bstore_u(rzo, __float_as_uint(zc + D), vz, 4 * (t0 + tt) * M);
                    const uint32_t ab = abs_bits(D), zb = abs_bits(zc);
                    emax = emax > ab ? emax : ab;
                    zmax = zmax > zb ? zmax : zb;
                }
            } else {
                // residual and masks of the tile (as in the forward pass)
                uint32_t mb = 0u;
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const int s = s0 + t0 + tt;
                    const float zt = (s == 0 || !forced) ? zprev : __fadd_rn(__fmul_rn(pi, zprev), __fmul_rn(alpha, rv[tt]));
                    const bool pos = zt > 0.f;
                    mb |= (pos ? 1u : 0u) << tt;
                    const float F = fmaf(Ai, zt, row16_dot(wr, pos ? zt : 0.f)) + hi;
                    zprev = zv[tt];
                    rv[tt] = zv[tt] - F;
                }
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool m = (mb >> tt) & 1u;
                    const float y = fmaf(d, D, row16_dot(wp, m ? D : 0.f));
                    D = fmaf(gm, y, -rv[tt]);
                    const float zc = zv[tt];
                    bstore_u(rzo, __float_as_uint(zc + D), vz, 4 * (t0 + tt) * M);
                    const uint32_t ab = abs_bits(D), zb = abs_bits(zc);
                    emax = emax > ab ? emax : ab;
                    zmax = zmax > zb ? zmax : zb;
                }
            }
        } else {
            for (int t = t0; t < t0 + tl; ++t) {
                const bool run = t < len && lat;
                const int s = s0 + t;
                const size_t step = (size_t)b * T + s;
                float zc = 0.f, xb = 0.f;
                if (run) {
                    zc = zin[step * M + c];
                    if (forced && s > 0) xb = x[((size_t)b * (T + 1) + s) * N + c];
                }
                float zt = 0.f;
                if (run) zt = (s == 0 || !forced) ? zprev : forced_in<WU>(pi, alpha, zprev, xb, s, tw);
                const bool pos = zt > 0.f;
                const float F = fmaf(Ai, zt, row16_dot(wr, pos ? zt : 0.f)) + hi;
                const float rc = zc - F;
                float Do = D;
                if constexpr (WU) Do = (forced && s <= tw) ? 0.f : D;
                const float y = fmaf(d, Do, row16_dot(wp, (run && pos) ? Do : 0.f));
                if (run) {
                    D = fmaf(gm, y, -rc);
                    zout[step * M + c] = zc + D;
                    const uint32_t ab = abs_bits(D), zb = abs_bits(zc);
                    emax = emax > ab ? emax : ab;
                    zmax = zmax > zb ? zmax : zb;
                    zprev = zc;
                }
            }
        }
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
        const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
        emax = emax > o ? emax : o;
        zmax = zmax > oz ? zmax : oz;
    }
    if (!fc.seq) {
        if (len > 0 && c == 0) {   // per-chain maxima, reduced per sequence by k_seq_max / k_seq_ctl
            chain_bits[id] = emax;
            chain_bits[(size_t)nchains + id] = zmax;
        }
        return;
    }
    // fused pass-end control: lane 0 gathers the four chains' maxima and arrives once per
    // sequence they belong to
    uint32_t em[4], zm[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        em[n] = (uint32_t)__shfl((int)emax, 16 * n, 64);
        zm[n] = (uint32_t)__shfl((int)zmax, 16 * n, 64);
    }
    if (lane == 0) {
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            const int bn = (chain0 + n) / ncs;
            if (w.plen[n] == 0 || (n > 0 && w.plen[n - 1] > 0 && (chain0 + n - 1) / ncs == bn)) continue;
            uint32_t E = 0u, Z = 0u;
            int cnt = 0;
#pragma unroll
            for (int m = n; m < 4; ++m)
                if (w.plen[m] > 0 && (chain0 + m) / ncs == bn) {
                    E = E > em[m] ? E : em[m];
                    Z = Z > zm[m] ? Z : zm[m];
                    ++cnt;
                }
            seq_arrive(fc, bn, cnt, ncs, E, Z);
        }
    }
}

// ---------------------------------------------------------------------------------------
// One kernel per Newton pass (M <= 16).  Where every sequence is a whole number of blocks of 32
// chunks of whole tiles, the fix-up of pass p and the forward pass of update p + 1 run in one
// kernel: a wave walks the group maps to its carry, takes its four chunks through pass p's
// update (z + Delta written out and kept in registers), and then forms the chunk products and
// chunk-local solutions of the next update on the new iterate, so the tile is loaded once and
// the start-up of the second kernel (control words, weights, tile loads) disappears.
// The next update is formed before the sequence's decision on pass p is known, with the
// damping an accepted update leads to; the decision stores in nd.pv that the aggregates belong
// to the new iterate only when the update is kept and the sequence goes on.  A sequence
// without valid aggregates (the first kernel, or after a rejected update) runs only the
// forward pass on its current iterate in the next kernel.  Aggregates alternate between two
// buffers (the kernel reads one and writes the other).
// The forward pass of a chunk needs the new iterate at the step before it.  Inside a wave it
// comes from the row before; for a wave's first chunk it is z + Delta with Delta the chunk's
// carry, and the previous wave puts exactly that value at its last step (it forms the next
// wave's carry with the same operations on the same operands instead of taking the end of its
// own recurrence, the same Delta to rounding), so no wave waits for another.
// ---------------------------------------------------------------------------------------
template <int TB, bool WU>
__global__ __launch_bounds__(512) void k_newton_pass16(
    const float *__restrict__ A, const float *__restrict__ W, const float *__restrict__ h, float alpha, int N,
    const float *__restrict__ x, const float *__restrict__ z0, float *zbuf, float *zalt, int T, int M, int C, int ncs,
    const float *__restrict__ Pin, const float *__restrict__ vin, const float *__restrict__ gin,
    float *__restrict__ Pout, float *__restrict__ vout, float *__restrict__ gout, FusedCtl fc, uint32_t *mark,
    uint32_t pass_no, int tw) {
    constexpr int WPB = 8;
    const int lane = threadIdx.x & 63, wvb = rfl_i((int)(threadIdx.x >> 6)), g = lane >> 4, c = lane & 15;
    if (mark && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(mark, pass_no, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const NewtonDev &nd = fc.nd;
    // a block's 32 chunks belong to one sequence b
    const int chain0 = (blockIdx.x * WPB + wvb) * 4;
    const int b = chain0 / ncs, cc0 = chain0 - b * ncs;
    if (nd.act[b] == 0) return;   // the whole block
    const bool have = nd.pv[b] == pass_no;
    const int sel = nd.sel[b];
    const float gam = nd.gamma[b];
    float omn = nd.om[b];   // the damping of the next update if this one is kept
    if (omn > 0.f) omn = omn / fc.dp.shrink < fc.dp.floor ? 0.f : omn / fc.dp.shrink;
    const float gnext = have ? 1.f - omn : gam;
    float *const zc = sel ? zalt : zbuf;   // current iterate
    float *const zn = sel ? zbuf : zalt;   // the update's output
    const int s0 = (cc0 + g) * C;          // first step of this lane's chunk
    const bool lat = c < M, forced = c < N;
    bool fr[4];   // B-operand rows 4 g + q of observed latents (dropped in warm-up steps)
#pragma unroll
    for (int q = 0; q < 4; ++q) fr[q] = 4 * g + q < N;
    const size_t row0 = (size_t)b * T + (size_t)cc0 * C, xrow0 = (size_t)b * (T + 1) + (size_t)cc0 * C;
    const auto rzc = wave_rsrc(zc + row0 * M), rzn = wave_rsrc(zn + row0 * M);
    const auto rx = wave_rsrc(N > 0 ? x + xrow0 * N : zc);
    const uint32_t vz = lat ? 4u * ((uint32_t)(g * C) * M + c) : kOffLane;
    const uint32_t vx = forced ? 4u * ((uint32_t)(g * C) * N + c) : kOffLane;
    // the first tile's loads go out first; the weights come through LDS (one load per element
    // for the block instead of gathers by every wave)
    float zv[TB], xv[TB];
#pragma unroll
    for (int tt = 0; tt < TB; ++tt) {
        zv[tt] = bload(rzc, vz, 4 * tt * M);
        xv[tt] = bload(rx, vx, 4 * tt * N);
    }
    float zprev = 0.f;   // z_{s0-1} of the current iterate (the initial state at s0 = 0)
    if (lat) {
        if (s0 == 0) zprev = z0 ? z0[(size_t)b * M + c] : (forced ? x[(size_t)b * (T + 1) * N + c] : 0.f);
        else zprev = zc[((size_t)b * T + s0 - 1) * M + c];
    }
    __shared__ float sW[256], sA[16], sH[16];
    {
        const int t = threadIdx.x;
        if (t < M * M) sW[t] = W[t];
        if (t < M) {
            sA[t] = A[t];
            sH[t] = h ? h[t] : 0.f;
        }
    }
    lds_barrier();
    int src[16];
    row_sources(c, src);
    float wr[16], wp[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        wr[k] = (lat && src[k] < M) ? sW[c * M + src[k]] : 0.f;
        wp[k] = wr[k] * p_of(src[k], N, alpha);
    }
    const float Ai = lat ? sA[c] : 0.f, hi = lat ? sH[c] : 0.f;
    const float pi = p_of(c, N, alpha), di = Ai * pi;
    float WpD[4], Dq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int col = 4 * g + q;
        const float wpq = (c < M && col < M) ? sW[c * M + col] * p_of(col, N, alpha) : 0.f;
        Dq[q] = (col == c && col < M) ? sA[col] * p_of(col, N, alpha) : 0.f;
        WpD[q] = wpq + Dq[q];
    }
    // ---- fix-up of the current update: the carry of this lane's chunk ----
    float D = 0.f, Dnext = 0.f;
    bool nextc = false;   // this lane's chunk ends where the next wave's starts
    if (have) {
        const int ngm = ncs / 32, grp = cc0 / 32;
        const float *Gb = gin + (size_t)b * ngm * 272;
        v4f cur = {0.f, 0.f, 0.f, 0.f};
        constexpr int PF = 4;
        float ga[PF][4], gv[PF][4];
        if (grp > 0) {
#pragma unroll
            for (int d2 = 0; d2 < PF; ++d2) {
                const float *Gk = Gb + (size_t)min(d2, grp - 1) * 272;
                carry16_fetch<false>(Gk, Gk + 256, g, c, ga[d2], gv[d2]);
            }
        }
        for (int k0 = 0; k0 < grp; k0 += PF) {
#pragma unroll
            for (int d2 = 0; d2 < PF; ++d2) {
                if (k0 + d2 >= grp) break;
                v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) nx = mfma16x16x4(ga[d2][q], cur[q], nx);
                if (c == 0) {
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2) nx[r2] += gv[d2][r2];
                }
                cur = nx;
                const float *Gk = Gb + (size_t)min(k0 + d2 + PF, grp - 1) * 272;
                carry16_fetch<false>(Gk, Gk + 256, g, c, ga[d2], gv[d2]);
            }
        }
        // the wave's carry: its prefix within the group (slot chain0) applied to the group's
        // carry; element k sits in lane 16 (k / 4), register k % 4, and is read as a scalar
        float wa[4], wvv[4];
        carry16_fetch<false>(Pin + (size_t)chain0 * 256, vin + (size_t)chain0 * 16, g, c, wa, wvv);
        v4f wc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < 4; ++q) wc = mfma16x16x4(wa[q], cur[q], wc);
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) wc[r2] += wvv[r2];
        float wk[16];
#pragma unroll
        for (int k = 0; k < 16; ++k)
            wk[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wc[k & 3]), 16 * (k >> 2)));
        if (g == 0) {
            float dv = wk[0];
#pragma unroll
            for (int k = 1; k < 16; ++k) dv = c == k ? wk[k] : dv;
            D = dv;
        } else {   // chunk g of the wave: R_g carry(wave) + s_g
            const float4 *R4 = reinterpret_cast<const float4 *>(Pin + (size_t)(chain0 + g) * 256 + c * 16);
            float a0 = vin[(size_t)(chain0 + g) * 16 + c], a1 = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 rr4 = R4[q];
                a0 = fmaf(rr4.x, wk[4 * q], a0);
                a1 = fmaf(rr4.y, wk[4 * q + 1], a1);
                a0 = fmaf(rr4.z, wk[4 * q + 2], a0);
                a1 = fmaf(rr4.w, wk[4 * q + 3], a1);
            }
            D = a0 + a1;
        }
        if (!lat) D = 0.f;
        // The carry of the next wave's first chunk, formed with the same operations on the same
        // operands as that wave forms it (one more group step when it starts the next group),
        // so both waves put the same z + Delta at the step between them.
        if (cc0 + 4 < ncs) {
            v4f curn = cur;
            if ((cc0 + 4) / 32 != grp) {
                float ga1[4], gv1[4];
                carry16_fetch<false>(Gb + (size_t)grp * 272, Gb + (size_t)grp * 272 + 256, g, c, ga1, gv1);
                v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) nx = mfma16x16x4(ga1[q], curn[q], nx);
                if (c == 0) {
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2) nx[r2] += gv1[r2];
                }
                curn = nx;
            }
            float wa2[4], wv2[4];
            carry16_fetch<false>(Pin + (size_t)(chain0 + 4) * 256, vin + (size_t)(chain0 + 4) * 16, g, c, wa2, wv2);
            v4f wcn = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) wcn = mfma16x16x4(wa2[q], curn[q], wcn);
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) wcn[r2] += wv2[r2];
            float dn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wcn[0]), 0));
#pragma unroll
            for (int kk = 1; kk < 16; ++kk) {
                const float e = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wcn[kk & 3]), 16 * (kk >> 2)));
                dn = c == kk ? e : dn;
            }
            if (g == 3 && lat) Dnext = dn;
            nextc = g == 3;
        }
    }
    // z_{s0-1} of the iterate the next update is formed at
    float zpn = have ? zprev + D : zprev;
    uint32_t emax = 0u, zmax = 0u;
    if (have) {
        // residual and masks at the current iterate, then Delta_t = gamma J~_t Delta_{t-1} - r_t;
        // the new iterate is written out and, in the last tile, kept in zv
        for (int t0 = 0; t0 < C; t0 += TB) {
            if (t0 > 0) {
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    zv[tt] = bload(rzc, vz, 4 * (t0 + tt) * M);
                    xv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);
                }
            }
            // a tile holding latent warm-up steps runs the body with P_1 in those steps
            bool wtile = false;
            if constexpr (WU) wtile = cc0 * C + t0 <= tw;
            if (wtile) {
                const uint32_t wb = low_bits(tw - (s0 + t0) + 1);   // bit tt: s0 + t0 + tt <= tw
                const uint32_t wf = forced ? wb : 0u;
                float rv[TB];
                uint32_t mb = 0u;
    #pragma unroll
                for (int tt = 0; tt < TB; tt += 2) {
                    const int s = s0 + t0 + tt;
                    const float zt0 = (s == 0 || !forced) ? zprev : forced_at<true>(pi, alpha, zprev, xv[tt], wb, tt);
                    const float zt1 = !forced ? zv[tt] : forced_at<true>(pi, alpha, zv[tt], xv[tt + 1], wb, tt + 1);
                    const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                    mb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                    float d0, d1;
                    row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                    rv[tt] = zv[tt] - (fmaf(Ai, zt0, d0) + hi);
                    rv[tt + 1] = zv[tt + 1] - (fmaf(Ai, zt1, d1) + hi);
                    zprev = zv[tt + 1];
                }
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool m = (mb >> tt) & 1u;
                    const float Do = ((wf >> tt) & 1u) ? 0.f : D;   // P_1: observed entries dropped
                    const float y = fmaf(di, Do, row16_dot(wp, m ? Do : 0.f));
                    D = fmaf(gam, y, -rv[tt]);
                    const float zcur = zv[tt];
                    // the last step before the next wave: its Delta as that wave's carry
                    const float dap = (tt == TB - 1 && t0 + TB == C && nextc) ? Dnext : D;
                    const float znew = zcur + dap;
                    if (t0 + TB < C) bstore_u(rzn, __float_as_uint(znew), vz, 4 * (t0 + tt) * M);
                    const uint32_t ab = lat ? abs_bits(dap) : 0u, zb = abs_bits(zcur);
                    emax = emax > ab ? emax : ab;
                    zmax = zmax > zb ? zmax : zb;
                    zv[tt] = znew;
                }
            } else {
                float rv[TB];
                uint32_t mb = 0u;
    #pragma unroll
                for (int tt = 0; tt < TB; tt += 2) {
                    const int s = s0 + t0 + tt;
                    const float zt0 = (s == 0 || !forced) ? zprev : __fadd_rn(__fmul_rn(pi, zprev), __fmul_rn(alpha, xv[tt]));
                    const float zt1 = !forced ? zv[tt] : __fadd_rn(__fmul_rn(pi, zv[tt]), __fmul_rn(alpha, xv[tt + 1]));
                    const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                    mb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                    float d0, d1;
                    row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                    rv[tt] = zv[tt] - (fmaf(Ai, zt0, d0) + hi);
                    rv[tt + 1] = zv[tt + 1] - (fmaf(Ai, zt1, d1) + hi);
                    zprev = zv[tt + 1];
                }
    #pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const bool m = (mb >> tt) & 1u;
                    const float y = fmaf(di, D, row16_dot(wp, m ? D : 0.f));
                    D = fmaf(gam, y, -rv[tt]);
                    const float zcur = zv[tt];
                    // the last step before the next wave: its Delta as that wave's carry
                    const float dap = (tt == TB - 1 && t0 + TB == C && nextc) ? Dnext : D;
                    const float znew = zcur + dap;
                    if (t0 + TB < C) bstore_u(rzn, __float_as_uint(znew), vz, 4 * (t0 + tt) * M);
                    const uint32_t ab = lat ? abs_bits(dap) : 0u, zb = abs_bits(zcur);
                    emax = emax > ab ? emax : ab;
                    zmax = zmax > zb ? zmax : zb;
                    zv[tt] = znew;
                }
            }
        }
        // z_{s0-1} of the new iterate exactly as stored: chunks 1..3 of the wave take it from the
        // row before; the first chunk's own carry equals the previous wave's (see above)
        const float zlast = __shfl(zv[TB - 1], (lane - 16) & 63, 64);
        if (g > 0) zpn = zlast;
        // the last tile of the new iterate; chunks of several tiles read it back
#pragma unroll
        for (int tt = 0; tt < TB; ++tt) bstore_u(rzn, __float_as_uint(zv[tt]), vz, 4 * (C - TB + tt) * M);
        if (C > TB) __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "agent");
    }
    // ---- the next update's forward pass ----
    const auto rzp = have ? rzn : rzc;   // the iterate it is formed at
    v4f acc[4];
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[n][r] = (4 * g + r == c) ? 1.f : 0.f;
    float u = 0.f;
    float gp = 1.f;   // gnext^TB: the damping of a tile's chunk product
#pragma unroll
    for (int k = 0; k < TB; ++k) gp *= gnext;
    for (int t0 = 0; t0 < C; t0 += TB) {
        if (C > TB && (have || t0 > 0)) {
#pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                zv[tt] = bload(rzp, vz, 4 * (t0 + tt) * M);
                xv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);
            }
        }
        bool wtile = false;   // a tile holding latent warm-up steps: P_1 in those steps
        if constexpr (WU) wtile = cc0 * C + t0 <= tw;
        if (wtile) {
            const uint32_t wb = low_bits(tw - (s0 + t0) + 1);   // bit tt: s0 + t0 + tt <= tw
            const uint32_t wf = forced ? wb : 0u;
            int lim[4];   // chain n: tile steps tt < lim[n] are warm-up steps
#pragma unroll
            for (int n = 0; n < 4; ++n) lim[n] = tw - ((cc0 + n) * C + t0) + 1;
            // residual and masks; r overwrites zv
            uint32_t posb = 0u;
    #pragma unroll
            for (int tt = 0; tt < TB; tt += 2) {
                const int s = s0 + t0 + tt;
                const float zt0 = (s == 0 || !forced) ? zpn : forced_at<true>(pi, alpha, zpn, xv[tt], wb, tt);
                const float zt1 = !forced ? zv[tt] : forced_at<true>(pi, alpha, zv[tt], xv[tt + 1], wb, tt + 1);
                const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                posb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                float d0, d1;
                row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                const float F0 = fmaf(Ai, zt0, d0) + hi, F1 = fmaf(Ai, zt1, d1) + hi;
                zpn = zv[tt + 1];
                zv[tt] = zv[tt] - F0;
                zv[tt + 1] = zv[tt + 1] - F1;
            }
    #pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                const bool pos = (posb >> tt) & 1u;
                const uint64_t bal = __ballot(pos);
                float Am[4][4];
    #pragma unroll
                for (int n = 0; n < 4; ++n)
    #pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                        Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                    }
                v4f nx[4];
    #pragma unroll
                for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                for (int q = 0; q < 4; ++q)
    #pragma unroll
                    for (int n = 0; n < 4; ++n)
                        nx[n] = mfma16x16x4(Am[n][q], (fr[q] && tt < lim[n]) ? 0.f : acc[n][q], nx[n]);
    #pragma unroll
                for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                const float uo = ((wf >> tt) & 1u) ? 0.f : u;
                const float y = fmaf(di, uo, row16_dot(wr, pos ? pi * uo : 0.f));
                u = fmaf(gnext, y, -zv[tt]);
            }
        } else {
            // residual and masks; r overwrites zv
            uint32_t posb = 0u;
    #pragma unroll
            for (int tt = 0; tt < TB; tt += 2) {
                const int s = s0 + t0 + tt;
                const float zt0 = (s == 0 || !forced) ? zpn : __fadd_rn(__fmul_rn(pi, zpn), __fmul_rn(alpha, xv[tt]));
                const float zt1 = !forced ? zv[tt] : __fadd_rn(__fmul_rn(pi, zv[tt]), __fmul_rn(alpha, xv[tt + 1]));
                const bool p0 = zt0 > 0.f, p1 = zt1 > 0.f;
                posb |= ((p0 ? 1u : 0u) | (p1 ? 2u : 0u)) << tt;
                float d0, d1;
                row16_dot2(wr, p0 ? zt0 : 0.f, p1 ? zt1 : 0.f, d0, d1);
                const float F0 = fmaf(Ai, zt0, d0) + hi, F1 = fmaf(Ai, zt1, d1) + hi;
                zpn = zv[tt + 1];
                zv[tt] = zv[tt] - F0;
                zv[tt + 1] = zv[tt + 1] - F1;
            }
    #pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                const bool pos = (posb >> tt) & 1u;
                const uint64_t bal = __ballot(pos);
                float Am[4][4];
    #pragma unroll
                for (int n = 0; n < 4; ++n)
    #pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                        Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                    }
                v4f nx[4];
    #pragma unroll
                for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                for (int q = 0; q < 4; ++q)
    #pragma unroll
                    for (int n = 0; n < 4; ++n) nx[n] = mfma16x16x4(Am[n][q], acc[n][q], nx[n]);
    #pragma unroll
                for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                const float y = fmaf(di, u, row16_dot(wr, pos ? pi * u : 0.f));
                u = fmaf(gnext, y, -zv[tt]);
            }
        }
        if (gnext != 1.f) {
#pragma unroll
            for (int n = 0; n < 4; ++n)
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) acc[n][r2] *= gp;
        }
    }
    if (!lat) u = 0.f;
    // ---- pass-end control of the current update (once per wave: its chunks share b) ----
    if (have) {
        emax = wave_max_u32(emax);
        zmax = wave_max_u32(zmax);
        if (lane == 0) seq_arrive(fc, b, 4, ncs, emax, zmax, pass_no + 1u);
    } else if (lane == 0) {
        // aggregates of the current iterate (nothing else of this sequence runs in this kernel)
        nd.pv[b] = pass_no + 1u;
    }
    // ---- wave maps and group maps of the next update (as in k_newton_product_plrnn16) ----
    __shared__ float lt[WPB][3][16][17];
    __shared__ float lv[WPB][4][16];
#pragma unroll
    for (int n = 1; n < 4; ++n)
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) lt[wvb][n - 1][4 * g + r2][c] = acc[n][r2];
    lv[wvb][g][c] = u;
    wave_lds_sync();   // each wave's own slots
    float Am[3][4];
    v4f bv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int n = 1; n < 4; ++n) Am[n - 1][q] = lt[wvb][n - 1][c][4 * g + q];
#pragma unroll
        for (int n = 0; n < 4; ++n) bv[n][q] = c == 0 ? lv[wvb][n][4 * g + q] : 0.f;
    }
    v4f R2 = {0.f, 0.f, 0.f, 0.f}, R3 = {0.f, 0.f, 0.f, 0.f}, Qw = {0.f, 0.f, 0.f, 0.f};
    v4f s2 = bv[1], s3 = bv[2], uw = bv[3];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        R2 = mfma16x16x4(Am[0][q], acc[0][q], R2);
        s2 = mfma16x16x4(Am[0][q], bv[0][q], s2);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        R3 = mfma16x16x4(Am[1][q], R2[q], R3);
        s3 = mfma16x16x4(Am[1][q], s2[q], s3);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        Qw = mfma16x16x4(Am[2][q], R3[q], Qw);
        uw = mfma16x16x4(Am[2][q], s3[q], uw);
    }
    const v4f outm[3] = {acc[0], R2, R3}, outv[3] = {bv[0], s2, s3};
#pragma unroll
    for (int n = 1; n < 4; ++n) {
        float *P = Pout + (size_t)(chain0 + n) * 256;
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = outm[n - 1][r2];
        if (c == 0)
            *reinterpret_cast<float4 *>(vout + (size_t)(chain0 + n) * 16 + 4 * g) =
                make_float4(outv[n - 1][0], outv[n - 1][1], outv[n - 1][2], outv[n - 1][3]);
    }
    __shared__ float lq[WPB][16][17];
    __shared__ float lu[WPB][16];
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) lq[wvb][4 * g + r2][c] = Qw[r2];
    if (c == 0) {
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) lu[wvb][4 * g + r2] = uw[r2];
    }
    __syncthreads();
    if (wvb != 0) return;
    const int bc0 = blockIdx.x * WPB * 4;   // the block's first chain
    v4f Gm, gu = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) Gm[r2] = (4 * g + r2 == c) ? 1.f : 0.f;
    for (int k = 0; k < WPB; ++k) {
        float *P = Pout + (size_t)(bc0 + 4 * k) * 256;
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = Gm[r2];
        if (c == 0)
            *reinterpret_cast<float4 *>(vout + (size_t)(bc0 + 4 * k) * 16 + 4 * g) =
                make_float4(gu[0], gu[1], gu[2], gu[3]);
        v4f ng = {0.f, 0.f, 0.f, 0.f}, nu;
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) nu[r2] = c == 0 ? lu[k][4 * g + r2] : 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float aq = lq[k][c][4 * g + q];
            ng = mfma16x16x4(aq, Gm[q], ng);
            nu = mfma16x16x4(aq, gu[q], nu);
        }
        Gm = ng;
        gu = nu;
    }
    const int ngm = ncs / (4 * WPB);
    float *Gp = gout + ((size_t)b * ngm + cc0 / (4 * WPB)) * 272;
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) Gp[(4 * g + r2) * 16 + c] = Gm[r2];
    if (c == 0) *reinterpret_cast<float4 *>(Gp + 256 + 4 * g) = make_float4(gu[0], gu[1], gu[2], gu[3]);
}

// ---------------------------------------------------------------------------------------
// The same forward Newton pass for M = 64 when every latent has the same forcing factor p
// (N = 0 or N = M).  Then the forced Jacobian factors as
//   J~_t = gp (diag(A) + W diag(m_t)),   gp = gamma p,
// so W itself (unscaled, in LDS) serves the matrix-core A operand, the residual F and the
// chunk-local solution, and no M x M operand lives in registers: the kernel fits two waves per
// SIMD, and one wave's VALU/LDS phase overlaps the other's matrix-core phase.  The scalar gp
// is applied to the chunk product every 8 steps (acc *= gp^8) instead of every step.
// One chain per wave (64 lanes = 64 latents for the lane-per-row part).
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ float lds_row_dot64(const float (*wl)[68], int row, const float *vec) {
    const float4 *w4 = reinterpret_cast<const float4 *>(wl[row]);
    const float4 *v4 = reinterpret_cast<const float4 *>(vec);
    float a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int q = 0; q < 16; q += 2) {
        const float4 w0 = w4[q], x0 = v4[q], w1 = w4[q + 1], x1 = v4[q + 1];
        a0 = fmaf(w0.x, x0.x, a0); a0 = fmaf(w0.y, x0.y, a0); a0 = fmaf(w0.z, x0.z, a0); a0 = fmaf(w0.w, x0.w, a0);
        a1 = fmaf(w1.x, x1.x, a1); a1 = fmaf(w1.y, x1.y, a1); a1 = fmaf(w1.z, x1.z, a1); a1 = fmaf(w1.w, x1.w, a1);
    }
    return a0 + a1;
}

// M = 64 with a uniform forcing factor (every latent forced, or none): one chain per wave, two
// waves per SIMD.  J_F = diag(A) + W diag(m) is the matrix-core A operand: W + diag(A) is staged in
// LDS once, and every step masks its columns with the step's ReLU bits (a column k of W is kept
// where m_k = 1; the diagonal entry becomes A_k where m_k = 0), one row tile of 16 at a time,
// shared by the four column tiles.  The chunk product alternates between two accumulator sets
// (the previous step's set is the unmasked B operand), so no copy, mask or scaling of the
// accumulators is needed per step; the factor gamma p is applied every 8 steps.  The residual
// and the chunk-local solution are row dot products against the same LDS rows, corrected for
// the diagonal: F_i = (W + diag A)_i relu(z~) + A_i min(z~_i, 0), and
// y_i = (W + diag A)_i (m o u) + A_i u_i (1 - m_i).
template <bool WU>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) void k_newton_product_plrnn64u(
    const float *__restrict__ A, const float *__restrict__ W, const float *__restrict__ h, float alpha, int N,
    const float *__restrict__ x, const float *__restrict__ z0, const float *zbuf, const float *zalt,
    const int *__restrict__ zsel, float *__restrict__ r_out, uint32_t *__restrict__ masks, float *__restrict__ Pout,
    float *__restrict__ vout, const int *__restrict__ active, const float *__restrict__ gamma, int B, int T, int M, int C,
    int ncs, int tw) {
    constexpr int MP = 64, NI = 4;
    __shared__ __align__(16) float wl[MP][68];   // W + diag(A), zero padded
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int id = blockIdx.x;
    const bool ok0 = id < B * ncs;
    const int b = ok0 ? id / ncs : 0, s0 = ok0 ? (id % ncs) * C : 0;
    const bool ok = ok0 && (!active || active[b]);
    const int len = ok ? min(C, T - s0) : 0;
    for (int e = lane; e < MP * MP; e += 64) {
        const int row = e / MP, col = e % MP;
        wl[row][col] = (row < M && col < M) ? W[row * M + col] + (row == col ? A[row] : 0.f) : 0.f;
    }
    const float p = N > 0 ? __fsub_rn(1.0f, alpha) : 1.0f;
    const float gp = (gamma ? gamma[b] : 1.f) * p;
    const float gp2 = gp * gp, gp4 = gp2 * gp2, gp8 = gp4 * gp4;
    // latent warm-up with every latent observed (N = M): the Jacobians of steps s <= tw are zero
    // (P_1 = 0), so a chunk that holds one has P = 0 (the product runs unchanged and is zeroed at
    // the end) and u restarts from -r there; N = 0 has no observed latent and no change
    const bool warmchunk = WU && N > 0 && s0 <= tw;
    // diagonal entries of this lane's A fragments: row 16 I + c is column 16 I + 4 g + q where
    // c == 4 g + q; there the masked entry is A instead of 0
    uint32_t dgA[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            dgA[I][q] = (c == 4 * g + q && 16 * I + c < M) ? __float_as_uint(A[16 * I + c]) : 0u;
    v4f acc[NI][4], acc2[NI][4];
#pragma unroll
    for (int Jt = 0; Jt < 4; ++Jt)
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[I][Jt][r] = (16 * I + 4 * g + r == 16 * Jt + c) ? 1.f : 0.f;
    // lane-per-row part: lane = latent
    const int ui = lane;
    const bool lat = ui < M;
    const float Ai = lat ? A[ui] : 0.f, hi = (lat && h) ? h[ui] : 0.f;
    const bool forced = ui < N;
    const float *z = cur_iter(zbuf, zalt, zsel, b);
    float zprev = 0.f;
    if (len > 0 && lat) {
        if (s0 == 0) zprev = z0 ? z0[(size_t)b * M + ui] : (forced ? x[(size_t)b * (T + 1) * N + ui] : 0.f);
        else zprev = z[((size_t)b * T + s0 - 1) * M + ui];
    }
    float u = 0.f;
    float zn = 0.f, xn = 0.f;
    if (len > 0 && lat) {
        zn = z[((size_t)b * T + s0) * M + ui];
        if (forced) xn = x[((size_t)b * (T + 1) + s0) * N + ui];
    }
    lds_barrier();   // W + diag(A) in LDS
    const int maxlen = __builtin_amdgcn_readfirstlane(len);
    // one step of the chain product, from accumulator set `in` to set `out`
    auto product = [&](const v4f (&in)[NI][4], v4f (&out)[NI][4], uint32_t w0, uint32_t w1) {
        uint32_t mk[4][4];   // all ones where the ReLU of column 16 j + 4 g + q is on
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                mk[j][q] = (uint32_t)__builtin_amdgcn_sbfe((int)((j >> 1) ? w1 : w0), 16 * (j & 1) + 4 * g + q, 1);
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            float a[4][4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float4 a4 = *reinterpret_cast<const float4 *>(&wl[16 * I + c][16 * j + 4 * g]);
                const float av[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t wb = __float_as_uint(av[q]);
                    // (m & (W + A delta)) | (~m & A delta): the diagonal tile keeps A where m = 0
                    a[j][q] = __uint_as_float(j == I ? ((mk[j][q] & wb) | (~mk[j][q] & dgA[I][q])) : (mk[j][q] & wb));
                }
            }
#pragma unroll
            for (int Jt = 0; Jt < 4; ++Jt) {
                v4f s = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) s = mfma16x16x4(a[j][q], in[j][Jt][q], s);
                out[I][Jt] = s;
            }
        }
    };
    auto step = [&](int t, const v4f (&in)[NI][4], v4f (&out)[NI][4]) {
        const bool run = lat;
        const int s = s0 + t;
        const float zcur = zn, xb = xn;
        if (t + 1 < len && lat) {
            zn = z[((size_t)b * T + s + 1) * M + ui];
            if (forced) xn = x[((size_t)b * (T + 1) + s + 1) * N + ui];
        }
        float zt = 0.f;
        if (run) {
            if (s == 0 || !forced) zt = zprev;
            else zt = forced_in<WU>(p, alpha, zprev, xb, s, tw);
        }
        const bool pos = zt > 0.f;
        const uint64_t bal = __ballot(pos);
        lds[lane] = pos ? zt : 0.f;
        lds_barrier();
        const float F = fmaf(Ai, fminf(zt, 0.f), lds_row_dot64(wl, ui, lds)) + hi;
        lds_barrier();
        const float r = zcur - F;
        if (run) {
            r_out[((size_t)b * T + s) * M + ui] = r;
            if (ui == 0) {
                const size_t stp = (size_t)b * T + s;
                masks[stp * 2] = (uint32_t)bal;
                if (M > 32) masks[stp * 2 + 1] = (uint32_t)(bal >> 32);
            }
        }
        // P <- (diag(A) + W diag(m)) P   (the factor gp is applied every 8 steps)
        product(in, out, (uint32_t)bal, (uint32_t)(bal >> 32));
        if ((t & 7) == 7) {
#pragma unroll
            for (int Jt = 0; Jt < 4; ++Jt)
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2) out[I][Jt][r2] *= gp8;
        }
        // chunk-local solution: u <- gp (A o u + W (m o u)) - r
        lds[lane] = pos ? u : 0.f;
        lds_barrier();
        const float y = fmaf(Ai, pos ? 0.f : u, lds_row_dot64(wl, ui, lds));
        lds_barrier();
        if (run) {
            const float gps = (warmchunk && s <= tw) ? 0.f : gp;   // J~_s = 0 in a warm-up step
            u = fmaf(gps, y, -r);
            zprev = zcur;
        }
    };
    int t = 0;
    for (; t + 1 < maxlen; t += 2) {
        step(t, acc, acc2);
        step(t + 1, acc2, acc);
    }
    if (t < maxlen) {   // odd length: the last step lands in the second set
        step(t, acc, acc2);
#pragma unroll
        for (int Jt = 0; Jt < 4; ++Jt)
#pragma unroll
            for (int I = 0; I < NI; ++I) acc[I][Jt] = acc2[I][Jt];
    }
    if (ok0 && len > 0) {
        float rest = warmchunk ? 0.f : 1.f;
        for (int k = 0; k < (len & 7); ++k) rest *= gp;
        float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
        for (int Jt = 0; Jt < 4; ++Jt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) P[(16 * I + 4 * g + r2) * MP + 16 * Jt + c] = acc[I][Jt][r2] * rest;
    }
    if (ok0) vout[(size_t)id * MP + ui] = u;
}

// ---------------------------------------------------------------------------------------
// carries across chunks
//   forward: carry_in[c] = y_end(c-1),  y_end(c) = P_c y_end(c-1) + v_c
//   reverse: carry_in[c] = lam_{s1(c)}, lam_{s0(c)} = P_c^T lam_{s1(c)} + v_c
// In processing order k (k = c forward, c = ncs - 1 - k reverse) both read
//   carry_in[c(k)] = cur_k,  cur_{k+1} = A_k cur_k + v_{c(k)},  A_k = P_c or P_c^T.
// Long chunk sequences use two levels: groups of G consecutive k are composed into one map
// (Q_j, u_j) (k_carry_group, all groups in parallel), the group carries are walked serially
// (k_carry over the groups), and every group re-walks its chunks from its carry (k_carry with
// a start vector).  Serial depth G + ncs / G + G instead of ncs.
// ---------------------------------------------------------------------------------------
template <int MP, bool REV>
__global__ __launch_bounds__(MP) void k_carry(const float *__restrict__ P, const float *__restrict__ v,
                                              float *__restrict__ carry_in, const int *__restrict__ active,
                                              uint32_t *__restrict__ norm_bits, int B, int ncs, int G,
                                              const float *__restrict__ start) {
    __shared__ __align__(16) float cs[MP];
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups, i = threadIdx.x;
    if (norm_bits && j == 0 && i == 0) {   // [0, B): max|Delta|, [B, 2B): max|z| of the next fix-up
        norm_bits[b] = 0u;
        norm_bits[B + b] = 0u;
    }
    if (active && !active[b]) return;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    float cur = start ? start[((size_t)b * ngroups + j) * MP + i] : 0.f;
    float pr[MP], pn[MP];
    auto load = [&](int step, float *dst) {
        const int cc = REV ? ncs - 1 - step : step;
        const float *Pc = P + ((size_t)b * ncs + cc) * MP * MP;
        if (!REV) {
            const float4 *r4 = reinterpret_cast<const float4 *>(Pc + i * MP);
#pragma unroll
            for (int q = 0; q < MP / 4; ++q) {
                float4 t = r4[q];
                dst[4 * q] = t.x; dst[4 * q + 1] = t.y; dst[4 * q + 2] = t.z; dst[4 * q + 3] = t.w;
            }
        } else {
#pragma unroll
            for (int k = 0; k < MP; ++k) dst[k] = Pc[k * MP + i];
        }
    };
    load(k0, pr);
    for (int step = k0; step < k1; ++step) {
        const int cc = REV ? ncs - 1 - step : step;
        const size_t id = (size_t)b * ncs + cc;
        if (step + 1 < k1) load(step + 1, pn);
        const float vv = v[id * MP + i];
        carry_in[id * MP + i] = cur;
        cs[i] = cur;
        lds_barrier();
        float a0 = vv, a1 = 0.f;
#pragma unroll
        for (int k = 0; k < MP; k += 2) {
            a0 = fmaf(pr[k], cs[k], a0);
            a1 = fmaf(pr[k + 1], cs[k + 1], a1);
        }
        lds_barrier();
        cur = a0 + a1;
#pragma unroll
        for (int k = 0; k < MP; ++k) pr[k] = pn[k];
    }
}

// group maps in processing order: Q_j = A_{k1-1} ... A_{k0}, u_j = the group's walk from 0
template <int MP, bool REV>
__global__ __launch_bounds__(256) void k_carry_group(const float *__restrict__ P, const float *__restrict__ v,
                                                     float *__restrict__ gq, float *__restrict__ gu,
                                                     const int *__restrict__ active, int ncs, int G) {
    constexpr int E = (MP * MP + 255) / 256;
    __shared__ float Q[MP][MP + 1], Am[MP][MP + 1], u[MP], vv[MP];
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups, tid = threadIdx.x;
    if (active && !active[b]) return;
    for (int e = tid; e < MP * MP; e += 256) Q[e / MP][e % MP] = (e / MP == e % MP) ? 1.f : 0.f;
    if (tid < MP) u[tid] = 0.f;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    // the next step's matrix and vector are loaded while this step is composed
    float pn[E], vn = 0.f;
    auto fetch = [&](int step) {
        const int cc = REV ? ncs - 1 - step : step;
        const float *Pc = P + ((size_t)b * ncs + cc) * MP * MP;
#pragma unroll
        for (int t = 0; t < E; ++t) {
            const int e = tid + 256 * t;
            pn[t] = (step < k1 && e < MP * MP) ? Pc[e] : 0.f;
        }
        vn = (step < k1 && tid < MP) ? v[((size_t)b * ncs + cc) * MP + tid] : 0.f;
    };
    fetch(k0);
    for (int step = k0; step < k1; ++step) {
#pragma unroll
        for (int t = 0; t < E; ++t) {
            const int e = tid + 256 * t;
            if (e < MP * MP) {
                const int r = e / MP, col = e % MP;
                if (REV) Am[col][r] = pn[t];
                else Am[r][col] = pn[t];
            }
        }
        if (tid < MP) vv[tid] = vn;
        fetch(step + 1);
        lds_barrier();
        float qn[E];
#pragma unroll
        for (int t = 0; t < E; ++t) {
            const int e = tid + 256 * t;
            float acc = 0.f;
            if (e < MP * MP) {
                const int r = e / MP, col = e % MP;
#pragma unroll(MP <= 32 ? MP : 8)
                for (int k = 0; k < MP; ++k) acc = fmaf(Am[r][k], Q[k][col], acc);
            }
            qn[t] = acc;
        }
        float un = 0.f;
        if (tid < MP) {
            un = vv[tid];
#pragma unroll
            for (int k = 0; k < MP; ++k) un = fmaf(Am[tid][k], u[k], un);
        }
        lds_barrier();
#pragma unroll
        for (int t = 0; t < E; ++t) {
            const int e = tid + 256 * t;
            if (e < MP * MP) Q[e / MP][e % MP] = qn[t];
        }
        if (tid < MP) u[tid] = un;
        lds_barrier();
    }
    float *q = gq + ((size_t)b * ngroups + j) * MP * MP;
    for (int e = tid; e < MP * MP; e += 256) q[e] = Q[e / MP][e % MP];
    if (tid < MP) gu[((size_t)b * ngroups + j) * MP + tid] = u[tid];
}

// ---------------------------------------------------------------------------------------
// M <= 16 carries on the matrix cores, one wave per walk.  A map A_k (P_c or its transpose)
// is the A operand of four 16x16x4 MFMAs; the vector being walked is column 0 of the B
// operand, whose accumulator layout is again the next step's B operand, so a step is four
// dependent MFMAs and no LDS.  The maps of the next PF steps are in flight while a step runs.
// ---------------------------------------------------------------------------------------

// walk of the vector: carry_in[c(k)] = cur_k, cur_{k+1} = A_k cur_k + v_{c(k)} (see k_carry)
template <bool REV>
__global__ __launch_bounds__(64) void k_carry16(const float *__restrict__ P, const float *__restrict__ v,
                                               float *__restrict__ carry_in, const int *__restrict__ active,
                                               uint32_t *__restrict__ norm_bits, int B, int ncs, int G,
                                               const float *__restrict__ start) {
    constexpr int PF = 8;
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups;
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    if (norm_bits && j == 0 && lane == 0) {   // [0, B): max|Delta|, [B, 2B): max|z| of the next fix-up
        norm_bits[b] = 0u;
        norm_bits[B + b] = 0u;
    }
    if (active && !active[b]) return;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    v4f cur;   // column 0: lane (g, 0) holds rows 4g..4g+3; other columns stay zero
#pragma unroll
    for (int r = 0; r < 4; ++r) cur[r] = (start && c == 0) ? start[((size_t)b * ngroups + j) * 16 + 4 * g + r] : 0.f;
    auto chunk = [&](int step) { return REV ? ncs - 1 - step : step; };
    float a[PF][4], vv[PF][4];
#pragma unroll
    for (int d = 0; d < PF; ++d) {
        const int cc = chunk(min(k0 + d, k1 - 1));
        carry16_fetch<REV>(P + ((size_t)b * ncs + cc) * 256, v + ((size_t)b * ncs + cc) * 16, g, c, a[d], vv[d]);
    }
    for (int k = k0; k < k1; k += PF) {
#pragma unroll
        for (int d = 0; d < PF; ++d) {
            const int step = k + d;
            if (step >= k1) break;
            const size_t id = (size_t)b * ncs + chunk(step);
            if (c == 0) *reinterpret_cast<float4 *>(carry_in + id * 16 + 4 * g) = make_float4(cur[0], cur[1], cur[2], cur[3]);
            v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) nx = mfma16x16x4(a[d][q], cur[q], nx);
            if (c == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) nx[r] += vv[d][r];
            }
            cur = nx;
            const int cn = chunk(min(step + PF, k1 - 1));
            carry16_fetch<REV>(P + ((size_t)b * ncs + cn) * 256, v + ((size_t)b * ncs + cn) * 16, g, c, a[d], vv[d]);
        }
    }
}

// group maps in processing order: Q_j = A_{k1-1} ... A_{k0}, u_j = the group's walk from 0
template <bool REV>
__global__ __launch_bounds__(64) void k_carry_group16(const float *__restrict__ P, const float *__restrict__ v,
                                                     float *__restrict__ gq, float *__restrict__ gu,
                                                     const int *__restrict__ active, int ncs, int G) {
    constexpr int PF = 8;
    const int ngroups = (ncs + G - 1) / G;
    const int b = blockIdx.x / ngroups, j = blockIdx.x % ngroups;
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    if (active && !active[b]) return;
    const int k0 = j * G, k1 = min(k0 + G, ncs);
    v4f Q, u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) Q[r] = (4 * g + r == c) ? 1.f : 0.f;
    auto chunk = [&](int step) { return REV ? ncs - 1 - step : step; };
    float a[PF][4], vv[PF][4];
#pragma unroll
    for (int d = 0; d < PF; ++d) {
        const int cc = chunk(min(k0 + d, k1 - 1));
        carry16_fetch<REV>(P + ((size_t)b * ncs + cc) * 256, v + ((size_t)b * ncs + cc) * 16, g, c, a[d], vv[d]);
    }
    for (int k = k0; k < k1; k += PF) {
#pragma unroll
        for (int d = 0; d < PF; ++d) {
            const int step = k + d;
            if (step >= k1) break;
            v4f nq = {0.f, 0.f, 0.f, 0.f}, nu = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                nq = mfma16x16x4(a[d][q], Q[q], nq);
                nu = mfma16x16x4(a[d][q], u[q], nu);
            }
            if (c == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) nu[r] += vv[d][r];
            }
            Q = nq;
            u = nu;
            const int cn = chunk(min(step + PF, k1 - 1));
            carry16_fetch<REV>(P + ((size_t)b * ncs + cn) * 256, v + ((size_t)b * ncs + cn) * 16, g, c, a[d], vv[d]);
        }
    }
    float *q = gq + ((size_t)b * ngroups + j) * 256;
#pragma unroll
    for (int r = 0; r < 4; ++r) q[(4 * g + r) * 16 + c] = Q[r];
    if (c == 0)
        *reinterpret_cast<float4 *>(gu + ((size_t)b * ngroups + j) * 16 + 4 * g) = make_float4(u[0], u[1], u[2], u[3]);
}

// d[k] += v(row_src(lane, k)) * s for k = 0..15: the rank-one update of a rotated row, e.g.
// dW[i][row_src(i, k)] += lam_i relu(z~)_{row_src(i, k)}.  All 64 lanes must be active.
#define DEER_RR(k) " row_ror:" #k " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
__device__ __forceinline__ void row16_outer(float (&d)[16], float v, float s) {
    asm volatile(
        "s_nop 1\n"
        "v_fmac_f32_e32 %0, %16, %17\n"
        "v_fmac_f32_dpp %1, %16, %17" DEER_RR(1)
        "v_fmac_f32_dpp %2, %16, %17" DEER_RR(2)
        "v_fmac_f32_dpp %3, %16, %17" DEER_RR(3)
        "v_fmac_f32_dpp %4, %16, %17" DEER_RR(4)
        "v_fmac_f32_dpp %5, %16, %17" DEER_RR(5)
        "v_fmac_f32_dpp %6, %16, %17" DEER_RR(6)
        "v_fmac_f32_dpp %7, %16, %17" DEER_RR(7)
        "v_fmac_f32_dpp %8, %16, %17" DEER_RR(8)
        "v_fmac_f32_dpp %9, %16, %17" DEER_RR(9)
        "v_fmac_f32_dpp %10, %16, %17" DEER_RR(10)
        "v_fmac_f32_dpp %11, %16, %17" DEER_RR(11)
        "v_fmac_f32_dpp %12, %16, %17" DEER_RR(12)
        "v_fmac_f32_dpp %13, %16, %17" DEER_RR(13)
        "v_fmac_f32_dpp %14, %16, %17" DEER_RR(14)
        "v_fmac_f32_dpp %15, %16, %17" DEER_RR(15)
        : "+v"(d[0]), "+v"(d[1]), "+v"(d[2]), "+v"(d[3]), "+v"(d[4]), "+v"(d[5]), "+v"(d[6]), "+v"(d[7]), "+v"(d[8]),
          "+v"(d[9]), "+v"(d[10]), "+v"(d[11]), "+v"(d[12]), "+v"(d[13]), "+v"(d[14]), "+v"(d[15])
        : "v"(v), "v"(s));
}
#undef DEER_RR

// ---------------------------------------------------------------------------------------
// M <= 16 reverse (adjoint) pass, per chunk [s0, s1) (gradients appendix):
//   P_c = J~_{s1} ... J~_{s0+1} over the steps below T (the carry pass takes its transpose)
//   v_c = lam_{s0} from lam_{s1} = 0,   lam_k = J~_{k+1}^T lam_{k+1} + g_k
// The masks m_s = [z~_s > 0] are formed here from z and x.  A tile row tt is chunk row
// t0 + tt: z_{s0+t0+tt}, x_{s0+t0+tt+1} (so z~ of step s0+t0+tt+1, the mask lam_k needs) and
// g_{s0+t0+tt}.  The products run forward over the tiles, the local adjoint backward.
// ---------------------------------------------------------------------------------------
template <int TB, bool WU>
__global__ __launch_bounds__(64) void k_chunk_product_plrnn16_rev(
    const float *__restrict__ A, const float *__restrict__ W, float alpha, int N, const float *__restrict__ rhs,
    const float *__restrict__ z, const float *__restrict__ x, float seed_scale, float *__restrict__ Pout,
    float *__restrict__ vout, int B, int T, int M, int C, int ncs, int wmaps, int tw) {
    static_assert(!WU || TB <= 16, "the warm-up variant runs 16-step tiles");
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * 4;
    const Chains16 w = chains16(chain0, nchains, ncs, C, T, nullptr, nullptr, nullptr);
    if (w.maxlen == 0) return;
    int pl[4];   // product steps: a chunk that ends at T has one fewer
    int minP = C;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const int s1 = ((chain0 + n) % ncs) * C + w.plen[n];
        pl[n] = w.plen[n] - ((w.plen[n] > 0 && s1 == T) ? 1 : 0);
        minP = min(minP, pl[n]);
    }
    float WpD[4], Dq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int col = 4 * g + q;
        const float wp = (c < M && col < M) ? W[c * M + col] * p_of(col, N, alpha) : 0.f;
        Dq[q] = (col == c && col < M) ? A[col] * p_of(col, N, alpha) : 0.f;
        WpD[q] = wp + Dq[q];
    }
    v4f acc[4];
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[n][r] = (4 * g + r == c) ? 1.f : 0.f;
    const int id = chain0 + g;
    const bool okc = id < nchains;
    int b, s0;
    chain_pos(chain0, g, nchains, ncs, C, b, s0);
    int len = 0;
#pragma unroll
    for (int n = 0; n < 4; ++n)
        if (n == g) len = w.plen[n];
    const bool lat = c < M, forced = c < N;
    bool fr[4];   // B-operand rows 4 g + q of observed latents (dropped in warm-up steps)
#pragma unroll
    for (int q = 0; q < 4; ++q) fr[q] = 4 * g + q < N;
    int src[16];
    row_sources(c, src);
    float wT[16];   // rotated row c of W^T
#pragma unroll
    for (int k = 0; k < 16; ++k) wT[k] = (lat && src[k] < M) ? W[src[k] * M + c] : 0.f;
    const float pi = p_of(c, N, alpha), Ai = lat ? A[c] : 0.f;
    const int b0 = chain0 / ncs, s00 = (chain0 % ncs) * C;
    const size_t row0 = (size_t)b0 * T + s00, xrow0 = (size_t)b0 * (T + 1) + s00 + 1;
    const uint32_t drow = (uint32_t)((size_t)b * T + s0 - row0);
    const uint32_t dxrow = (uint32_t)((size_t)b * (T + 1) + s0 + 1 - xrow0);
    const auto rz = wave_rsrc(z + row0 * M), rg = wave_rsrc(rhs ? rhs + row0 * M : z);
    const auto rx = wave_rsrc(N > 0 ? x + xrow0 * N : z);
    const uint32_t vz = lat ? 4u * (drow * M + c) : kOffLane;
    const uint32_t vx = forced ? 4u * (dxrow * N + c) : kOffLane;
    const uint32_t vg = (rhs && lat) ? vz : kOffLane;
    float zv[TB], xv[TB];
    uint32_t posb = 0u;
    int loaded = -1;   // t0 of the tile whose rows zv/xv hold
    auto load_tile = [&](int t0) {
#pragma unroll
        for (int tt = 0; tt < TB; ++tt) {
            zv[tt] = bload(rz, vz, 4 * (t0 + tt) * M);
            xv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);
        }
        posb = 0u;
        uint32_t wb = 0u;   // bit tt: step s0 + t0 + tt + 1 is a latent warm-up step
        if constexpr (WU) wb = low_bits(tw - (s0 + t0));
#pragma unroll
        for (int tt = 0; tt < TB; ++tt) {
            const float zt = forced ? forced_at<WU>(pi, alpha, zv[tt], xv[tt], wb, tt) : zv[tt];
            posb |= (zt > 0.f ? 1u : 0u) << tt;
        }
        loaded = t0;
    };
    // z~ of step s = s0 + t + 1 for the slow path (chunk row t)
    auto ztilde_next = [&](int t) {
        if (!(t < len && lat)) return 0.f;
        const int s = s0 + t + 1;
        const float zp = z[((size_t)b * T + s - 1) * M + c];
        if (!forced) return zp;
        return forced_in<WU>(pi, alpha, zp, x[((size_t)b * (T + 1) + s) * N + c], s, tw);
    };
    // ---- chunk products, forward over the tiles
    for (int t0 = 0; t0 < w.maxlen; t0 += TB) {
        const int tl = min(TB, w.maxlen - t0);
        if (t0 + TB <= w.minlen) {
            load_tile(t0);
            if (t0 + TB <= minP) {
                bool wtile = false;   // some chain has a latent warm-up step in this tile
                if constexpr (WU) {
#pragma unroll
                    for (int n = 0; n < 4; ++n) wtile = wtile || w.cs[n] + t0 + 1 <= tw;
                }
                if (wtile) {
                    int lim[4];   // chain n: the steps of tile rows tt < lim[n] are warm-up steps
#pragma unroll
                    for (int n = 0; n < 4; ++n) lim[n] = tw - (w.cs[n] + t0);
    #pragma unroll
                    for (int tt = 0; tt < TB; ++tt) {
                        const uint64_t bal = __ballot((posb >> tt) & 1u);
                        float Am[4][4];
    #pragma unroll
                        for (int n = 0; n < 4; ++n)
    #pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const uint32_t m =
                                    (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                                Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                            }
                        v4f nx[4];
    #pragma unroll
                        for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                        for (int q = 0; q < 4; ++q)
    #pragma unroll
                            for (int n = 0; n < 4; ++n)
                                nx[n] = mfma16x16x4(Am[n][q], (fr[q] && tt < lim[n]) ? 0.f : acc[n][q], nx[n]);
    #pragma unroll
                        for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                    }
                } else {
    #pragma unroll
                    for (int tt = 0; tt < TB; ++tt) {
                        const uint64_t bal = __ballot((posb >> tt) & 1u);
                        float Am[4][4];
    #pragma unroll
                        for (int n = 0; n < 4; ++n)
    #pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const uint32_t m =
                                    (uint32_t)__builtin_amdgcn_sbfe((int)(uint32_t)(bal >> (16 * n)), 4 * g + q, 1);
                                Am[n][q] = __uint_as_float((m & __float_as_uint(WpD[q])) | (~m & __float_as_uint(Dq[q])));
                            }
                        v4f nx[4];
    #pragma unroll
                        for (int n = 0; n < 4; ++n) nx[n] = v4f{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                        for (int q = 0; q < 4; ++q)
    #pragma unroll
                            for (int n = 0; n < 4; ++n) nx[n] = mfma16x16x4(Am[n][q], acc[n][q], nx[n]);
    #pragma unroll
                        for (int n = 0; n < 4; ++n) acc[n] = nx[n];
                    }
                }
            } else {
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) {
                    const uint64_t bal = __ballot((posb >> tt) & 1u);
#pragma unroll
                    for (int n = 0; n < 4; ++n)
                        if (t0 + tt < pl[n]) {
                            if (WU && w.cs[n] + t0 + tt + 1 <= tw)
                                acc[n] = mfma_step16_warm(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq, fr);
                            else
                                acc[n] = mfma_step16(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq);
                        }
                }
            }
        } else {
            for (int t = t0; t < t0 + tl; ++t) {
                const uint64_t bal = __ballot(ztilde_next(t) > 0.f);
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    if (t < pl[n]) {
                        if (WU && w.cs[n] + t + 1 <= tw)
                            acc[n] = mfma_step16_warm(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq, fr);
                        else
                            acc[n] = mfma_step16(acc[n], (uint32_t)(bal >> (16 * n)), g, WpD, Dq);
                    }
            }
        }
    }
    // ---- local adjoint from a zero carry, backward over the tiles
    float u = 0.f;
    const int last = ((w.maxlen - 1) / TB) * TB;
    for (int t0 = last; t0 >= 0; t0 -= TB) {
        const int tl = min(TB, w.maxlen - t0);
        if (t0 + TB <= w.minlen) {
            if (loaded != t0) load_tile(t0);
            float gv[TB];
#pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                if (rhs) gv[tt] = bload(rg, vg, 4 * (t0 + tt) * M);
                else gv[tt] = forced ? seed_scale * (zv[tt] - xv[tt]) : 0.f;
            }
            // latent warm-up: no MSE seed for rows k < tw; P_{k+1} = P_1 drops the observed
            // latents' entries of J~_{k+1}^T lam for k + 1 <= tw
            uint32_t kill = 0u;
            if constexpr (WU) {
                const uint32_t wr2 = low_bits(tw - (s0 + t0));   // bit tt: row s0 + t0 + tt < tw
                if (!rhs) {
#pragma unroll
                    for (int tt = 0; tt < TB; ++tt) gv[tt] = ((wr2 >> tt) & 1u) ? 0.f : gv[tt];
                }
                kill = forced ? wr2 : 0u;   // same bits: s0 + t0 + tt + 1 <= tw
            }
#pragma unroll
            for (int tt = TB - 1; tt >= 0; --tt) {
                const bool m = (posb >> tt) & 1u;
                const float wt = row16_dot(wT, u);
                bool on = t0 + tt + 1 < len;   // J~_{k+1}^T, P_{k+1} on the left
                if constexpr (WU) on = on && !((kill >> tt) & 1u);
                const float y = on ? pi * fmaf(Ai, u, m ? wt : 0.f) : 0.f;
                if (lat) u = y + gv[tt];
            }
        } else {
            for (int t = t0 + tl - 1; t >= t0; --t) {
                const bool run = t < len && lat;
                const bool m = (t + 1 < len) && ztilde_next(t) > 0.f;
                const float wt = row16_dot(wT, u);
                if (run) {
                    const size_t step = (size_t)b * T + s0 + t;
                    bool on = t + 1 < len;
                    if constexpr (WU) on = on && !(forced && s0 + t + 1 <= tw);
                    const float y = on ? pi * fmaf(Ai, u, m ? wt : 0.f) : 0.f;
                    float gk = 0.f;
                    if (rhs) gk = rhs[step * M + c];
                    else if (forced && (!WU || s0 + t >= tw))
                        gk = seed_scale * (z[step * M + c] - x[((size_t)b * (T + 1) + s0 + t + 1) * N + c]);
                    u = y + gk;
                }
            }
        }
    }
    if (wmaps) {
        // Composed for the reverse carry pass (processing order c0+3, c0+2, c0+1, c0):
        //   slot chain0 + 3:      wave map  Q = (P_3 P_2 P_1 P_0)^T, u_w = the four chunks' walk
        //   slot chain0 + 3 - j:  prefix    R_j = (P_3 ... P_{4-j})^T, s_j, j = 1..3
        // so that carry(chain0 + 3 - j) = R_j carry(chain0 + 3) + s_j.  The accumulator layout of
        // P_n is the A-operand layout of P_n^T; P_3^T as a B operand comes through LDS.
        __shared__ float lt[16][17];
        __shared__ float lv[4][16];
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) lt[4 * g + r2][c] = acc[3][r2];
        lv[g][c] = u;
        lds_barrier();
        v4f R1, bv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            R1[q] = lt[c][4 * g + q];   // B layout of P_3^T
#pragma unroll
            for (int n = 0; n < 4; ++n) bv[n][q] = c == 0 ? lv[n][4 * g + q] : 0.f;
        }
        v4f R2 = {0.f, 0.f, 0.f, 0.f}, R3 = {0.f, 0.f, 0.f, 0.f}, Qw = {0.f, 0.f, 0.f, 0.f};
        v4f s2 = bv[2], s3 = bv[1], uw = bv[0];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            R2 = mfma16x16x4(acc[2][q], R1[q], R2);
            s2 = mfma16x16x4(acc[2][q], bv[3][q], s2);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            R3 = mfma16x16x4(acc[1][q], R2[q], R3);
            s3 = mfma16x16x4(acc[1][q], s2[q], s3);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            Qw = mfma16x16x4(acc[0][q], R3[q], Qw);
            uw = mfma16x16x4(acc[0][q], s3[q], uw);
        }
        // R1 = P_3^T in accumulator layout is the transposed store of acc[3]
        const v4f outm[4] = {R3, R2, R1, Qw}, outv[4] = {s3, s2, bv[3], uw};
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            float *P = Pout + (size_t)(chain0 + n) * 256;
            if (n == 2) {
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) P[c * 16 + 4 * g + r2] = acc[3][r2];
            } else {
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = outm[n][r2];
            }
            if (c == 0)
                *reinterpret_cast<float4 *>(vout + (size_t)(chain0 + n) * 16 + 4 * g) =
                    make_float4(outv[n][0], outv[n][1], outv[n][2], outv[n][3]);
        }
        return;
    }
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const int cid = chain0 + n;
        if (cid < nchains && w.plen[n] > 0) {
            float *P = Pout + (size_t)cid * 256;
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) P[(4 * g + r2) * 16 + c] = acc[n][r2];
        }
    }
    if (okc) vout[(size_t)id * 16 + c] = u;
}

// M <= 16 reverse fix-up: lam_k from the carry lam_{s1}, written out, with the parameter-
// gradient partial sums dW[i][j] += lam_i relu(z~_j), dA_i += lam_i z~_i, dh_i += lam_i over
// the wave's four chains (layout gpart[wave][16][18], the rotated dW columns put back).  A tile
// row tt is step k = s0 + t0 + tt: z_k, x_k, x_{k+1}, g_k, and z_{k-1} for z~_k.
template <int TB, bool WU>
__global__ __launch_bounds__(64) void k_fixup_rev_plrnn16(const float *__restrict__ A, const float *__restrict__ W,
                                                         float alpha, int N, const float *__restrict__ gin,
                                                         float seed_scale, const float *__restrict__ x,
                                                         const float *__restrict__ z0, const float *__restrict__ z,
                                                         const float *__restrict__ carry_in,
                                                         const float *__restrict__ Pm, const float *__restrict__ vmap,
                                                         float *__restrict__ lam_out, float *__restrict__ gpart, int B,
                                                         int T, int M, int C, int ncs, int tw) {
    static_assert(!WU || TB <= 16, "the warm-up variant runs 16-step tiles (bit masks of TB + 1 steps)");
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int nchains = B * ncs;
    const int chain0 = blockIdx.x * 4;
    const Chains16 w = chains16(chain0, nchains, ncs, C, T, nullptr, nullptr, nullptr);
    const int id = chain0 + g;
    const bool okc = id < nchains;
    int b, s0;
    chain_pos(chain0, g, nchains, ncs, C, b, s0);
    int len = 0;
#pragma unroll
    for (int n = 0; n < 4; ++n)
        if (n == g) len = w.plen[n];
    const bool lat = c < M, forced = c < N;
    int src[16];
    row_sources(c, src);
    float wT[16], dW[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        wT[k] = (lat && src[k] < M) ? W[src[k] * M + c] : 0.f;
        dW[k] = 0.f;
    }
    const float pi = p_of(c, N, alpha), Ai = lat ? A[c] : 0.f;
    float lam = 0.f, dA = 0.f, dh = 0.f;
    if (len > 0 && lat) {
        if (!Pm || g == 3) {
            lam = carry_in[(size_t)id * 16 + c];
        } else {   // composed wave maps: carry = R carry(chain0 + 3) + s
            const float4 *R4 = reinterpret_cast<const float4 *>(Pm + (size_t)id * 256 + c * 16);
            const float4 *w4 = reinterpret_cast<const float4 *>(carry_in + (size_t)(chain0 + 3) * 16);
            float a0 = vmap[(size_t)id * 16 + c], a1 = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 rr4 = R4[q], ww = w4[q];
                a0 = fmaf(rr4.x, ww.x, a0);
                a1 = fmaf(rr4.y, ww.y, a1);
                a0 = fmaf(rr4.z, ww.z, a0);
                a1 = fmaf(rr4.w, ww.w, a1);
            }
            lam = a0 + a1;
        }
    }
    // z~ of step s (array index) for this lane
    auto ztilde = [&](int s) {
        if (s == 0) return z0 ? z0[(size_t)b * M + c] : (forced ? x[(size_t)b * (T + 1) * N + c] : 0.f);
        const float zp = z[((size_t)b * T + s - 1) * M + c];
        if (!forced) return zp;
        return forced_in<WU>(pi, alpha, zp, x[((size_t)b * (T + 1) + s) * N + c], s, tw);
    };
    const int cl0 = min(chain0, nchains - 1);
    const int b0 = cl0 / ncs, s00 = (cl0 % ncs) * C;
    const size_t row0 = (size_t)b0 * T + s00, xrow0 = (size_t)b0 * (T + 1) + s00;
    const uint32_t drow = (uint32_t)((size_t)b * T + s0 - row0);
    const uint32_t dxrow = (uint32_t)((size_t)b * (T + 1) + s0 - xrow0);
    const auto rz = wave_rsrc(z + row0 * M), rg = wave_rsrc(gin ? gin + row0 * M : z);
    const auto rx = wave_rsrc(N > 0 ? x + xrow0 * N : z), rl = wave_rsrc(lam_out ? lam_out + row0 * M : z);
    const uint32_t vz = lat ? 4u * (drow * M + c) : kOffLane;
    const uint32_t vx = forced ? 4u * (dxrow * N + c) : kOffLane;
    const uint32_t vg = (gin && lat) ? vz : kOffLane, vl = (lam_out && lat) ? vz : kOffLane;
    const int last = w.maxlen > 0 ? ((w.maxlen - 1) / TB) * TB : -1;
    for (int t0 = last; t0 >= 0; t0 -= TB) {
        const int tl = min(TB, w.maxlen - t0);
        if (t0 + TB <= w.minlen) {
            float zv[TB], xv[TB + 1], gv[TB], zt[TB + 1];
#pragma unroll
            for (int tt = 0; tt < TB; ++tt) {
                zv[tt] = bload(rz, vz, 4 * (t0 + tt) * M);
                xv[tt] = bload(rx, vx, 4 * (t0 + tt) * N);
                gv[tt] = bload(rg, vg, 4 * (t0 + tt) * M);
            }
            xv[TB] = bload(rx, vx, 4 * (t0 + TB) * N);
            // z~ of steps s0+t0 .. s0+t0+TB (the last only for the mask of the tile's top step);
            // with a latent warm-up, bit j of wb marks step s0 + t0 + j <= tw (j <= TB <= 16)
            uint32_t wb = 0u;
            if constexpr (WU) wb = low_bits(tw - (s0 + t0) + 1);
            zt[0] = (len > 0 && lat) ? ztilde(s0 + t0) : 0.f;
#pragma unroll
            for (int tt = 1; tt <= TB; ++tt)
                zt[tt] = forced ? forced_at<WU>(pi, alpha, zv[tt - 1], xv[tt], wb, tt) : zv[tt - 1];
            if (!gin) {
#pragma unroll
                for (int tt = 0; tt < TB; ++tt) gv[tt] = forced ? seed_scale * (zv[tt] - xv[tt + 1]) : 0.f;
                if constexpr (WU) {   // no MSE seed for the warm-up rows k < tw
#pragma unroll
                    for (int tt = 0; tt < TB; ++tt) gv[tt] = ((wb >> (tt + 1)) & 1u) ? 0.f : gv[tt];
                }
            }
            const uint32_t kill = forced ? (wb >> 1) : 0u;   // bit tt: P_{k+1} = P_1 (k + 1 <= tw)
#pragma unroll
            for (int tt = TB - 1; tt >= 0; --tt) {
                const int k = s0 + t0 + tt;
                bool nxt = k + 1 < T;   // J~_{k+1}^T, P_{k+1} on the left
                if constexpr (WU) nxt = nxt && !((kill >> tt) & 1u);
                const bool m = zt[tt + 1] > 0.f;
                const float wt = row16_dot(wT, lam);
                const float y = nxt ? pi * fmaf(Ai, lam, m ? wt : 0.f) : 0.f;
                if (lat) lam = y + gv[tt];
                bstore_u(rl, __float_as_uint(lam), vl, 4 * (t0 + tt) * M);
                const float zk = lat ? zt[tt] : 0.f;
                dA = fmaf(lam, zk, dA);
                dh += lat ? lam : 0.f;
                row16_outer(dW, zk > 0.f ? zk : 0.f, lat ? lam : 0.f);
            }
        } else {
            for (int t = t0 + tl - 1; t >= t0; --t) {
                const bool run = t < len && lat;
                const int k = s0 + t;
                const bool nxt = run && k + 1 < T;
                const bool m = nxt && ztilde(k + 1) > 0.f;
                bool on = nxt;
                if constexpr (WU) on = on && !(forced && k + 1 <= tw);
                const float wt = row16_dot(wT, lam);
                float zk = 0.f, lr = 0.f;
                if (run) {
                    const size_t step = (size_t)b * T + k;
                    const float y = on ? pi * fmaf(Ai, lam, m ? wt : 0.f) : 0.f;
                    float gk = 0.f;
                    if (gin) gk = gin[step * M + c];
                    else if (forced && (!WU || k >= tw))
                        gk = seed_scale * (z[step * M + c] - x[((size_t)b * (T + 1) + k + 1) * N + c]);
                    lam = y + gk;
                    if (lam_out) lam_out[step * M + c] = lam;
                    zk = ztilde(k);
                    lr = lam;
                    dA = fmaf(lam, zk, dA);
                    dh += lam;
                }
                row16_outer(dW, zk > 0.f ? zk : 0.f, lr);
            }
        }
    }
    // sum over the wave's four chains and write the wave's partial
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
#pragma unroll
        for (int k = 0; k < 16; ++k) dW[k] += __shfl_xor(dW[k], off, 64);
        dA += __shfl_xor(dA, off, 64);
        dh += __shfl_xor(dh, off, 64);
    }
    if (g == 0) {
        float *gp = gpart + ((size_t)blockIdx.x * 16 + c) * 18;
#pragma unroll
        for (int k = 0; k < 16; ++k) gp[src[k]] = dW[k];
        gp[16] = dA;
        gp[17] = dh;
    }
}

// Carries of composed wave maps (four chunks each): one block per sequence, NWV waves.  Each
// wave composes a contiguous range of maps into one, wave 0 walks the NWV composed maps (LDS),
// and every wave walks its range again from its own carry, writing the carry of each wave map.
// Forward: map of wave w at chunk slot 4w, walked w = 0, 1, ...; reverse (adjoint): at slot
// 4w + 3, walked w = nw - 1, nw - 2, ...; the carry goes to the same slot as the map.
constexpr int WALK_NWV = 16;
template <bool REV>
__global__ __launch_bounds__(WALK_NWV * 64) void k_carry_walk16(const float *__restrict__ P, const float *__restrict__ v,
                                                               float *__restrict__ carry,
                                                               const int *__restrict__ active, int ncs) {
    constexpr int PF = 8;
    __shared__ float ls[WALK_NWV][16][17];
    __shared__ float lt[WALK_NWV][16], lsc[WALK_NWV][16];
    const int b = blockIdx.x;
    if (active && !active[b]) return;
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    const int nw = ncs >> 2, per = (nw + WALK_NWV - 1) / WALK_NWV;
    const int w0 = min(wv * per, nw), w1 = min(w0 + per, nw);
    const float *Pb = P + (size_t)b * ncs * 256, *vb = v + (size_t)b * ncs * 16;
    auto slot = [&](int k) { return REV ? 4 * (nw - 1 - k) + 3 : 4 * k; };   // processing position k
    auto fetch = [&](int k, float (&a)[4], float (&vv)[4]) {
        carry16_fetch<false>(Pb + (size_t)slot(k) * 256, vb + (size_t)slot(k) * 16, g, c, a, vv);
    };
    float a[PF][4], vv[PF][4];
    // composed map of this wave's range
    v4f S, t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) S[r] = (4 * g + r == c) ? 1.f : 0.f;
    if (w0 < w1) {
#pragma unroll
        for (int d = 0; d < PF; ++d) fetch(min(w0 + d, w1 - 1), a[d], vv[d]);
        for (int k = w0; k < w1; k += PF) {
#pragma unroll
            for (int d = 0; d < PF; ++d) {
                if (k + d >= w1) break;
                v4f ns = {0.f, 0.f, 0.f, 0.f}, nt = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    ns = mfma16x16x4(a[d][q], S[q], ns);
                    nt = mfma16x16x4(a[d][q], t[q], nt);
                }
                if (c == 0) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) nt[r] += vv[d][r];
                }
                S = ns;
                t = nt;
                if (per > PF) fetch(min(k + d + PF, w1 - 1), a[d], vv[d]);   // else kept for the re-walk
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) ls[wv][4 * g + r][c] = S[r];
    if (c == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) lt[wv][4 * g + r] = t[r];
    }
    __syncthreads();
    if (wv == 0) {   // walk of the composed maps
        v4f cur = {0.f, 0.f, 0.f, 0.f};
        for (int k = 0; k < WALK_NWV; ++k) {
            if (c == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) lsc[k][4 * g + r] = cur[r];
            }
            v4f nx;
#pragma unroll
            for (int r = 0; r < 4; ++r) nx[r] = c == 0 ? lt[k][4 * g + r] : 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) nx = mfma16x16x4(ls[k][c][4 * g + q], cur[q], nx);
            cur = nx;
        }
    }
    __syncthreads();
    if (w0 >= w1) return;
    v4f cur;
#pragma unroll
    for (int r = 0; r < 4; ++r) cur[r] = c == 0 ? lsc[wv][4 * g + r] : 0.f;
    if (per > PF) {
#pragma unroll
        for (int d = 0; d < PF; ++d) fetch(min(w0 + d, w1 - 1), a[d], vv[d]);
    }
    for (int k = w0; k < w1; k += PF) {
#pragma unroll
        for (int d = 0; d < PF; ++d) {
            const int wm = k + d;
            if (wm >= w1) break;
            if (c == 0)
                *reinterpret_cast<float4 *>(carry + ((size_t)b * ncs + slot(wm)) * 16 + 4 * g) =
                    make_float4(cur[0], cur[1], cur[2], cur[3]);
            v4f nx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) nx = mfma16x16x4(a[d][q], cur[q], nx);
            if (c == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) nx[r] += vv[d][r];
            }
            cur = nx;
            if (per > PF) fetch(min(wm + PF, w1 - 1), a[d], vv[d]);
        }
    }
}

// ---------------------------------------------------------------------------------------
// forward fix-up: Delta from the carry, z += Delta, per-sequence max |Delta|
// ---------------------------------------------------------------------------------------
template <int MP, bool WU>
__global__ __launch_bounds__(64) void k_fixup_fwd_plrnn(const float *__restrict__ A, const float *__restrict__ W,
                                                        float alpha, int N, const uint32_t *__restrict__ masks,
                                                        const float *__restrict__ r, const float *__restrict__ carry_in,
                                                        float *zbuf, float *zalt, const int *__restrict__ zsel,
                                                        uint32_t *__restrict__ chain_bits, const int *__restrict__ active,
                                                        const float *__restrict__ gamma, int B, int T, int M, int C,
                                                        int ncs, int tw) {
    using G = Geo<MP>;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * G::NCH + n;
    const bool ok0 = id < B * ncs;
    const int b = ok0 ? id / ncs : 0, cc = ok0 ? id % ncs : 0;
    const bool ok = ok0 && (!active || active[b]);
    const int s0 = cc * C, len = ok ? min(C, T - s0) : 0;
    const float gm = gamma ? gamma[b] : 1.f;
    const float *zin = cur_iter(zbuf, zalt, zsel, b);
    float *zout = next_iter(zbuf, zalt, zsel, b);
    float wrow[MP];
#pragma unroll
    for (int k = 0; k < MP; ++k) wrow[k] = (i < M && k < M) ? W[i * M + k] * p_of(k, N, alpha) : 0.f;
    const float d = i < M ? A[i] * p_of(i, N, alpha) : 0.f;
    float D = (ok && i < M) ? carry_in[(size_t)id * MP + i] : 0.f;
    uint32_t emax = 0u, zmax = 0u;
    const int maxlen = __builtin_amdgcn_readfirstlane(C);
    // the loads of a step are issued PD steps ahead
    auto fetch = [&](int t, float &rv, float &zv, uint32_t &mw) {
        const bool run = t < len && i < M;
        const size_t step = (size_t)b * T + s0 + t;
        rv = run ? r[step * M + i] : 0.f;
        zv = run ? zin[step * M + i] : 0.f;
        mw = run ? masks[step * G::MW + (i >> 5)] : 0u;
    };
    constexpr int PD = 2;
    float rq[PD], zq[PD];
    uint32_t mq[PD];
#pragma unroll
    for (int q = 0; q < PD; ++q) fetch(q, rq[q], zq[q], mq[q]);
    for (int t = 0; t < maxlen; ++t) {
        const bool run = t < len && i < M;
        const size_t step = (size_t)b * T + s0 + t;
        const float rc = rq[0], zc = zq[0];
        const uint32_t mc = mq[0];
#pragma unroll
        for (int q = 0; q + 1 < PD; ++q) {
            rq[q] = rq[q + 1];
            zq[q] = zq[q + 1];
            mq[q] = mq[q + 1];
        }
        fetch(t + PD, rq[PD - 1], zq[PD - 1], mq[PD - 1]);
        const float Do = (WU && i < N && s0 + t <= tw) ? 0.f : D;   // P_1 in a latent warm-up step
        lds[lane] = (run && ((mc >> (i & 31)) & 1u)) ? Do : 0.f;
        lds_barrier();
        const float y = fmaf(d, Do, lds_dot<MP>(lds, n, wrow));
        lds_barrier();
        if (run) {
            D = fmaf(gm, y, -rc);
            zout[step * M + i] = zc + D;
            const uint32_t ab = abs_bits(D), zb = abs_bits(zc);
            emax = emax > ab ? emax : ab;
            zmax = zmax > zb ? zmax : zb;
        }
    }
    // max over the MP lanes of this chain
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

// ---------------------------------------------------------------------------------------
// forward fix-up on the matrix cores (16 < M <= 64): a block runs 16 chains as the 16 columns,
// wave w owning the 16-row tile w of
//   y = W diag(p) (m o Delta) + (A p) o Delta,   Delta' = gamma y - r,   z' = z + Delta'
// A = rows 16w + c of W diag(p) (registers for the whole chunk); B = (m o Delta) of all latents
// of the 16 chains in the k-permuted layout (lane (g, c): latent 16j + 4g + q of chain c), read
// from LDS, where every wave puts its new tile each step (double-buffered: one barrier a step).
// The same update as k_fixup_fwd_plrnn, 16 MFMAs per wave and step instead of an M-long dot
// product per lane.
// ---------------------------------------------------------------------------------------
template <int MP, bool VEC, bool WU>
__global__ __launch_bounds__(MP * 4) void k_fixup_fwd_plrnn_mf(const float *__restrict__ A, const float *__restrict__ W,
                                                               float alpha, int N, const uint32_t *__restrict__ masks,
                                                               const float *__restrict__ r,
                                                               const float *__restrict__ carry_in, float *zbuf,
                                                               float *zalt, const int *__restrict__ zsel,
                                                               uint32_t *__restrict__ chain_bits,
                                                               const int *__restrict__ active,
                                                               const float *__restrict__ gamma, int B, int T, int M,
                                                               int C, int ncs, int tw) {
    using G = Geo<MP>;
    constexpr int NW = MP / 16, NS = MP / 4, DQ = MP + 4;
    __shared__ __align__(16) float dls[2][16 * DQ];   // [buffer][chain c][latent]
    __shared__ uint32_t mx[NW][16][2];
    const int tid = threadIdx.x, wv = rfl_i(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    float aw[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int k = 16 * (s / 4) + 4 * g + (s % 4), row = 16 * wv + c;
        aw[s] = (row < M && k < M) ? W[row * M + k] * p_of(k, N, alpha) : 0.f;
    }
    const int i0 = 16 * wv + 4 * g;   // this lane's output latents i0 .. i0 + 3 of chain c
    float dg[4];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) dg[rr] = i0 + rr < M ? A[i0 + rr] * p_of(i0 + rr, N, alpha) : 0.f;
    const int nchains = B * ncs;
    const int id = blockIdx.x * 16 + c;
    const bool exists = id < nchains;
    const int b = exists ? id / ncs : 0, cc = exists ? id % ncs : 0;
    const bool ok = exists && (!active || active[b]);
    const int s0 = cc * C;
    const int len = ok ? min(C, T - s0) : 0;
    int maxlen = len;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) maxlen = max(maxlen, __shfl_xor(maxlen, off, 64));
    maxlen = rfl_i(maxlen);
    const float gm = gamma ? gamma[b] : 1.f;
    const float *zin = cur_iter(zbuf, zalt, zsel, b);
    float *zout = next_iter(zbuf, zalt, zsel, b);
    constexpr bool vec = VEC;   // M % 4 == 0: whole 16-byte groups of latents
    const size_t rowb = (size_t)b * T + s0;
    {
        float4 d4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ok) {
            const float *ci = carry_in + (size_t)id * MP + i0;
            d4 = make_float4(i0 < M ? ci[0] : 0.f, i0 + 1 < M ? ci[1] : 0.f, i0 + 2 < M ? ci[2] : 0.f,
                             i0 + 3 < M ? ci[3] : 0.f);
        }
        *reinterpret_cast<float4 *>(&dls[0][c * DQ + i0]) = d4;
    }
    // step inputs a tile of PD steps at a time, double-buffered in registers: r and z of the
    // lane's four latents, the chain's mask words
    constexpr int PD = 8;
    float4 rq[PD], zq[PD];
    uint32_t mq0[PD], mq1[PD];
    // Branch-free: every lane loads from a valid address (a step past the chunk reads the chunk's
    // first row, a latent past M reads latent 0) and the values that do not apply are zeroed, so
    // the compiler counts the outstanding loads exactly and waits only for the step it consumes.
    auto fetch = [&](int t, float4 &rn, float4 &zn, uint32_t &mn0, uint32_t &mn1) {
        const bool run = t < len;
        const size_t row = rowb + (run ? t : 0);
        const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (vec) {
            const bool keep = run && i0 < M;
            const size_t e = row * M + (i0 < M ? i0 : 0);
            const float4 rv = *reinterpret_cast<const float4 *>(r + e);
            const float4 zv = *reinterpret_cast<const float4 *>(zin + e);
            rn = keep ? rv : z4;
            zn = keep ? zv : z4;
        } else {
            float rv[4], zv[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bool keep = run && i0 + q < M;
                const size_t e = row * M + (i0 + q < M ? i0 + q : 0);
                const float a = r[e], bz = zin[e];
                rv[q] = keep ? a : 0.f;
                zv[q] = keep ? bz : 0.f;
            }
            rn = make_float4(rv[0], rv[1], rv[2], rv[3]);
            zn = make_float4(zv[0], zv[1], zv[2], zv[3]);
        }
        const uint32_t w0 = masks[row * G::MW];
        const uint32_t w1 = G::MW > 1 ? masks[row * G::MW + 1] : 0u;
        mn0 = run ? w0 : 0u;
        mn1 = run ? w1 : 0u;
    };
#pragma unroll
    for (int u = 0; u < PD; ++u) fetch(u, rq[u], zq[u], mq0[u], mq1[u]);
    uint32_t emax = 0u, zmax = 0u;
    lds_barrier();
    for (int t0 = 0; t0 < maxlen; t0 += PD) {
        // the next tile's inputs go out now and are taken over after this tile's PD steps, so
        // the only wait for them falls there (not inside the steps)
        float4 rn2[PD], zn2[PD];
        uint32_t mn0b[PD], mn1b[PD];
#pragma unroll
        for (int u = 0; u < PD; ++u) fetch(t0 + PD + u, rn2[u], zn2[u], mn0b[u], mn1b[u]);
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            const int t = t0 + u;
            if (t >= maxlen) break;
            const int cur = u & 1;   // PD is even: buffer parity follows t
            const float4 rc = rq[u], zc = zq[u];
            const uint32_t m0 = mq0[u], m1 = mq1[u];
            float bv[NS];
            float4 own = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int j = 0; j < NS / 4; ++j) {
                const float4 dq = *reinterpret_cast<const float4 *>(&dls[cur][c * DQ + 16 * j + 4 * g]);
                if (j == wv) own = dq;
                const uint32_t w = (j >> 1) ? m1 : m0;
                const int sh = 16 * (j & 1) + 4 * g;
                bv[4 * j + 0] = select_bit(w, sh + 0, dq.x);
                bv[4 * j + 1] = select_bit(w, sh + 1, dq.y);
                bv[4 * j + 2] = select_bit(w, sh + 2, dq.z);
                bv[4 * j + 3] = select_bit(w, sh + 3, dq.w);
            }
            if constexpr (WU) {   // a latent warm-up step of chain c (P_1): observed entries of Delta dropped
                if (s0 + t <= tw) {
#pragma unroll
                    for (int k = 0; k < NS; ++k)
                        if (16 * (k / 4) + 4 * g + (k % 4) < N) bv[k] = 0.f;
                    own.x = i0 < N ? 0.f : own.x;
                    own.y = i0 + 1 < N ? 0.f : own.y;
                    own.z = i0 + 2 < N ? 0.f : own.z;
                    own.w = i0 + 3 < N ? 0.f : own.w;
                }
            }
            // two accumulators over alternate k-steps: half the dependent chain
            v4f acc = {0.f, 0.f, 0.f, 0.f}, acc2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < NS; k += 2) {
                acc = mfma16x16x4(aw[k], bv[k], acc);
                acc2 = mfma16x16x4(aw[k + 1], bv[k + 1], acc2);
            }
            const float dold[4] = {own.x, own.y, own.z, own.w};
            const float rr4[4] = {rc.x, rc.y, rc.z, rc.w}, zz4[4] = {zc.x, zc.y, zc.z, zc.w};
            float dn[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) dn[q] = fmaf(gm, fmaf(dg[q], dold[q], acc[q] + acc2[q]), -rr4[q]);
            if (t < len) {
                const size_t e = (rowb + t) * M + i0;
                if (vec) {
                    if (i0 < M)
                        *reinterpret_cast<float4 *>(zout + e) =
                            make_float4(zz4[0] + dn[0], zz4[1] + dn[1], zz4[2] + dn[2], zz4[3] + dn[3]);
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (i0 + q < M) zout[e + q] = zz4[q] + dn[q];
                }
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (i0 + q < M) {
                        const uint32_t ab = abs_bits(dn[q]), zb = abs_bits(zz4[q]);
                        emax = emax > ab ? emax : ab;
                        zmax = zmax > zb ? zmax : zb;
                    }
            }
            *reinterpret_cast<float4 *>(&dls[cur ^ 1][c * DQ + i0]) =
                make_float4(i0 < M ? dn[0] : 0.f, i0 + 1 < M ? dn[1] : 0.f, i0 + 2 < M ? dn[2] : 0.f,
                            i0 + 3 < M ? dn[3] : 0.f);
            lds_barrier();
        }
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            rq[u] = rn2[u];
            zq[u] = zn2[u];
            mq0[u] = mn0b[u];
            mq1[u] = mn1b[u];
        }
    }
    // per-chain maxima: the lane groups, then the waves
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
        const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
        emax = emax > o ? emax : o;
        zmax = zmax > oz ? zmax : oz;
    }
    if (g == 0) {
        mx[wv][c][0] = emax;
        mx[wv][c][1] = zmax;
    }
    lds_barrier();
    if (wv == 0 && g == 0 && ok) {   // reduced per sequence by the pass-end control
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            emax = emax > mx[w][c][0] ? emax : mx[w][c][0];
            zmax = zmax > mx[w][c][1] ? zmax : mx[w][c][1];
        }
        chain_bits[id] = emax;
        chain_bits[(size_t)nchains + id] = zmax;
    }
}

// per-sequence max over its chains of the bits the forward fix-ups left:
// norm_bits[b] = max |Delta|, norm_bits[B + b] = max |z| (unsigned max of |x| bits, NaN-propagating)
__global__ __launch_bounds__(256) void k_seq_max(const uint32_t *__restrict__ chain_bits, const int *__restrict__ active,
                                                 uint32_t *__restrict__ norm_bits, int B, int ncs) {
    __shared__ uint32_t red[2][4];
    const int b = blockIdx.x, tid = threadIdx.x;
    if (active && !active[b]) return;
    uint32_t e = 0u, zm = 0u;
    for (int c = tid; c < ncs; c += 256) {
        const uint32_t a = chain_bits[(size_t)b * ncs + c], z = chain_bits[(size_t)B * ncs + (size_t)b * ncs + c];
        e = e > a ? e : a;
        zm = zm > z ? zm : z;
    }
    e = wave_max_u32(e);
    zm = wave_max_u32(zm);
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = e;
        red[1][tid >> 6] = zm;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t a = red[0][0], z = red[1][0];
        for (int w = 1; w < 4; ++w) {
            a = a > red[0][w] ? a : red[0][w];
            z = z > red[1][w] ? z : red[1][w];
        }
        norm_bits[b] = a;
        norm_bits[B + b] = z;
    }
}

int launch_seq_max(const uint32_t *chain_bits, const int *active, uint32_t *norm_bits, int B, int ncs,
                   hipStream_t st) {
    KTimer kt("k_seq_max", st);
    hipLaunchKernelGGL(k_seq_max, dim3(B), dim3(256), 0, st, chain_bits, active, norm_bits, B, ncs);
    DEER_LAUNCH_CHECK("k_seq_max");
    return DEER_OK;
}

// Convergence test and update safeguard of one Newton pass, per sequence, on the device (so
// that passes are queued without a host round trip).  From the maxima of the pass's chains:
// accept the update (flip sel, count it, relax the damping, freeze the sequence once
// max|Delta| < tol), or reject it (keep sel, raise the damping: 1 - gamma = first, then x grow
// up to 1 = the fixed-point step); a non-finite fixed-point step ends the sequence.
__global__ __launch_bounds__(256) void k_seq_ctl(const uint32_t *__restrict__ chain_bits, NewtonDev nd, int B,
                                                 int ncs, float tol, float bound, NewtonDamp dp) {
    __shared__ uint32_t red[2][4];
    const int b = blockIdx.x, tid = threadIdx.x;
    if (!nd.act[b]) return;
    uint32_t e = 0u, zm = 0u;
    for (int c = tid; c < ncs; c += 256) {
        const uint32_t a = chain_bits[(size_t)b * ncs + c], z = chain_bits[(size_t)B * ncs + (size_t)b * ncs + c];
        e = e > a ? e : a;
        zm = zm > z ? zm : z;
    }
    e = wave_max_u32(e);
    zm = wave_max_u32(zm);
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = e;
        red[1][tid >> 6] = zm;
    }
    __syncthreads();
    if (tid != 0) return;
    for (int w = 1; w < 4; ++w) {
        e = e > red[0][w] ? e : red[0][w];
        zm = zm > red[1][w] ? zm : red[1][w];
    }
    seq_decide(b, e, zm, nd, tol, bound, dp);
}

int launch_seq_ctl(const uint32_t *chain_bits, const NewtonDev &nd, int B, int ncs, float tol, float bound,
                   const NewtonDamp &dp, hipStream_t st) {
    KTimer kt("k_seq_ctl", st);
    hipLaunchKernelGGL(k_seq_ctl, dim3(B), dim3(256), 0, st, chain_bits, nd, B, ncs, tol, bound, dp);
    DEER_LAUNCH_CHECK("k_seq_ctl");
    return DEER_OK;
}

__global__ void k_ctl_init(NewtonDev nd, uint32_t *seq, int B) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    if (seq) {
#pragma unroll
        for (int k = 0; k < 3; ++k) seq[(size_t)b * kSeqWords + 32 * k] = 0u;
    }
    nd.act[b] = 1;
    nd.gamma[b] = 1.f;
    nd.sel[b] = 0;
    nd.om[b] = 0.f;
    nd.it[b] = 0;
    nd.norm[b] = __uint_as_float(0x7fc00000u);
    nd.status[b] = 0;
    if (nd.pv) nd.pv[b] = 0u;   // no aggregates yet (pass numbers start at 1)
}

int launch_ctl_init(const NewtonDev &nd, uint32_t *seq, int B, hipStream_t st) {
    hipLaunchKernelGGL(k_ctl_init, dim3((B + 255) / 256), dim3(256), 0, st, nd, seq, B);
    DEER_LAUNCH_CHECK("k_ctl_init");
    return DEER_OK;
}

// ---------------------------------------------------------------------------------------
// reverse fix-up: lam from the carry, written out, with the parameter-gradient partial
// sums of this chunk: dW[i][j] += lam_i relu(z~_j), dA_i += lam_i z~_i, dh_i += lam_i
// (layout gpart[chain][MP][MP + 2]).
// ---------------------------------------------------------------------------------------
template <int MP, bool WU>
__global__ __launch_bounds__(64) void k_fixup_rev_plrnn(const float *__restrict__ A, const float *__restrict__ W,
                                                        float alpha, int N, const uint32_t *__restrict__ masks,
                                                        const float *__restrict__ gin, float seed_scale,
                                                        const float *__restrict__ x, const float *__restrict__ z0,
                                                        const float *__restrict__ z, const float *__restrict__ carry_in,
                                                        float *__restrict__ lam_out, float *__restrict__ gpart, int B,
                                                        int T, int M, int C, int ncs, int tw) {
    using G = Geo<MP>;
    __shared__ __align__(16) float lds[64];
    const int lane = threadIdx.x, n = lane / MP, i = lane % MP;
    const int id = blockIdx.x * G::NCH + n;
    const bool ok = id < B * ncs;
    const int b = ok ? id / ncs : 0, cc = ok ? id % ncs : 0;
    const int s0 = cc * C, s1 = ok ? min(s0 + C, T) : s0;
    float wcol[MP], dW[MP];
#pragma unroll
    for (int k = 0; k < MP; ++k) {
        wcol[k] = (i < M && k < M) ? W[k * M + i] : 0.f;
        dW[k] = 0.f;
    }
    const float pi = p_of(i, N, alpha), Ai = i < M ? A[i] : 0.f;
    float lam = (ok && i < M) ? carry_in[(size_t)id * MP + i] : 0.f;
    float dA = 0.f, dh = 0.f;
    const int maxlen = __builtin_amdgcn_readfirstlane(C);
    // per-step inputs (mask of step k + 1, cotangent g_k, forced state z~_{k-1}), PD steps ahead
    auto fetch = [&](int t, float &mv, float &gv, float &zv) {
        const int k = s1 - 1 - t;
        const bool run = k >= s0 && i < M;
        mv = 0.f;
        gv = 0.f;
        zv = 0.f;
        if (run) {
            const size_t step = (size_t)b * T + k;
            if (k + 1 < T) mv = (float)mask_bit(masks, step + 1, G::MW, i);
            if (gin) gv = gin[step * M + i];
            else if (i < N && (!WU || k >= tw))   // no MSE seed for the warm-up states
                gv = seed_scale * (z[step * M + i] - x[((size_t)b * (T + 1) + k + 1) * N + i]);
            zv = forced_state(x, z0, z, b, k, i, T, M, N, alpha, WU ? tw : 0);
        }
    };
    constexpr int PD = 1;
    float mq[PD], gq[PD], zq[PD];
#pragma unroll
    for (int q = 0; q < PD; ++q) fetch(q, mq[q], gq[q], zq[q]);
    for (int t = 0; t < maxlen; ++t) {
        const int k = s1 - 1 - t;
        const bool run = k >= s0 && i < M;
        const float mc = mq[0], gk = gq[0], zc = zq[0];
#pragma unroll
        for (int q = 0; q + 1 < PD; ++q) {
            mq[q] = mq[q + 1];
            gq[q] = gq[q + 1];
            zq[q] = zq[q + 1];
        }
        fetch(t + PD, mq[PD - 1], gq[PD - 1], zq[PD - 1]);
        lds[lane] = lam;
        lds_barrier();
        const float wt = lds_dot<MP>(lds, n, wcol);
        lds_barrier();
        float zt = 0.f;
        if (run) {
            const size_t step = (size_t)b * T + k;
            // J~_{k+1}^T lam, P_{k+1} = P_1 dropping the observed rows in a latent warm-up step
            const bool jon = k + 1 < T && !(WU && i < N && k + 1 <= tw);
            const float y = jon ? pi * fmaf(Ai, lam, mc * wt) : 0.f;
            lam = y + gk;
            if (lam_out) lam_out[step * M + i] = lam;
            zt = zc;
            dA = fmaf(lam, zt, dA);
            dh += lam;
        }
        const float lr = run ? lam : 0.f;
        lds[lane] = (run && zt > 0.f) ? zt : 0.f;
        lds_barrier();
        const float4 *l4 = reinterpret_cast<const float4 *>(lds + n * MP);
#pragma unroll
        for (int q = 0; q < MP / 4; ++q) {
            const float4 v = l4[q];
            dW[4 * q + 0] = fmaf(lr, v.x, dW[4 * q + 0]);
            dW[4 * q + 1] = fmaf(lr, v.y, dW[4 * q + 1]);
            dW[4 * q + 2] = fmaf(lr, v.z, dW[4 * q + 2]);
            dW[4 * q + 3] = fmaf(lr, v.w, dW[4 * q + 3]);
        }
        lds_barrier();
    }
    if (ok) {
        float *gp = gpart + ((size_t)id * MP + i) * (MP + 2);
#pragma unroll
        for (int k = 0; k < MP; ++k) gp[k] = dW[k];
        gp[MP] = dA;
        gp[MP + 1] = dh;
    }
}

// sum the per-chunk partials in float64 in two stages: blocks over (slice of the chains, 64
// consecutive entries of [MP][MP + 2]), the four waves of a block taking every fourth chain of
// the slice with 8 loads in flight and their sums added through LDS in a fixed order; then the
// slices
constexpr int GP_SLICES = 64;

__global__ __launch_bounds__(256) void k_reduce_gpart1(const float *__restrict__ gpart, int nchains, int n,
                                                       double *__restrict__ part2) {
    __shared__ double red[4][64];
    const int sl = blockIdx.x;
    const int c0 = (int)((long)nchains * sl / GP_SLICES), c1 = (int)((long)nchains * (sl + 1) / GP_SLICES);
    const int cg = threadIdx.x >> 6;
    const int e = blockIdx.y * 64 + (threadIdx.x & 63);
    const bool ok = e < n;
    double s0 = 0.0, s1 = 0.0;
    for (int ch0 = c0 + cg; ch0 < c1; ch0 += 32) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int ch = ch0 + 4 * k;
            v[k] = (ok && ch < c1) ? gpart[(size_t)ch * n + e] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < 8; k += 2) {
            s0 += (double)v[k];
            s1 += (double)v[k + 1];
        }
    }
    red[cg][threadIdx.x & 63] = s0 + s1;
    __syncthreads();
    if (cg != 0 || !ok) return;
    const int l = threadIdx.x & 63;
    part2[(size_t)sl * n + e] = (red[0][l] + red[1][l]) + (red[2][l] + red[3][l]);
}

__global__ __launch_bounds__(256) void k_reduce_gpart2(const double *__restrict__ part2, int MP, int M,
                                                       float *__restrict__ dA, float *__restrict__ dW,
                                                       float *__restrict__ dh) {
    const int n = MP * (MP + 2);
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= n) return;
    const int i = e / (MP + 2), j = e % (MP + 2);
    if (i >= M || (j < MP && j >= M)) return;
    double s = 0.0;
    for (int sl = 0; sl < GP_SLICES; ++sl) s += part2[(size_t)sl * n + e];
    const float v = (float)s;
    if (j < MP) {
        if (dW) dW[i * M + j] = v;
    } else if (j == MP) {
        if (dA) dA[i] = v;
    } else {
        if (dh) dh[i] = v;
    }
}

size_t reduce_gpart_ws_bytes(int MP) { return (size_t)GP_SLICES * MP * (MP + 2) * sizeof(double); }

// ---------------------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------------------
static int invalid_arg(const char *what) {
    set_error("%s", what);
    return DEER_ERR_INVALID_ARG;
}

static int padded(int M) { return M <= 16 ? 16 : (M <= 32 ? 32 : (M <= 64 ? 64 : 128)); }

// The ReLU masks of the vanilla PLRNN alone (m_t = z~_{t-1} > 0 per latent, the decision of
// k_resjac_plrnn without its residual): an elementwise pass over [B, T, M] for callers that need
// no F, r or J (the adjoint).  A wave holds RQ groups of 64 / MP rows (lane = latent) and issues
// their loads together; the (sequence, step) of the rows come from one division per pass.
template <int MP>
__global__ __launch_bounds__(256) void k_masks_plrnn(float alpha, int N, const float *__restrict__ x,
                                                     const float *__restrict__ z0, const float *__restrict__ z,
                                                     uint32_t *__restrict__ masks, const int *__restrict__ active,
                                                     int B, int T, int M, int tw) {
    constexpr int NCH = 64 / MP, RQ = 8;
    const int lane = threadIdx.x & 63, n = lane / MP, i = lane % MP;
    const long total = (long)B * T;
    const long gw = (long)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (long)gridDim.x * 4;
    constexpr long per = (long)NCH * RQ;
    for (long r0 = gw * per; r0 < total; r0 += nw * per) {
        const RowBase rb = row_base(r0, T);
        float zt[RQ];
        bool act[RQ];
#pragma unroll
        for (int q = 0; q < RQ; ++q) {
            const int rr = q * NCH + n;
            const bool in = r0 + rr < total;
            int b = 0, s = 0;
            if (in) row_at(rb, rr, T, b, s);
            act[q] = in && (!active || active[b]);
            zt[q] = (act[q] && i < M) ? forced_state(x, z0, z, b, s, i, T, M, N, alpha, tw) : 0.f;
        }
#pragma unroll
        for (int q = 0; q < RQ; ++q) {
            const uint64_t bal = __ballot(zt[q] > 0.f);
            const long row = r0 + q * NCH + n;
            if (act[q] && i == 0) {
                if (MP == 64) {
                    masks[(size_t)row * 2 + 0] = (uint32_t)bal;
                    if (M > 32) masks[(size_t)row * 2 + 1] = (uint32_t)(bal >> 32);
                } else {
                    const uint64_t seg = bal >> (n * MP);
                    masks[row] = (uint32_t)(MP == 32 ? seg : (seg & 0xffffull));
                }
            }
        }
    }
}

int launch_resjac_plrnn(const PlrnnArgs &a, const float *z, float *F, float *r, float *J, uint32_t *masks,
                        const int *active, hipStream_t st) {
    const int MP = padded(a.M);
    if (!F && !r && !J) {
        if (!masks) return DEER_OK;
        const long waves = ((long)a.B * a.T + (64 / MP) * 8 - 1) / ((64 / MP) * 8);
        const long want = (waves + 3) / 4;
        const int grid = (int)(want < 4096 ? want : 4096);
        KTimer kt("k_masks_plrnn", st);
        if (MP == 16)
            hipLaunchKernelGGL(k_masks_plrnn<16>, dim3(grid), dim3(256), 0, st, a.alpha, a.N, a.x, a.z0, z, masks, active, a.B, a.T, a.M, a.tw);
        else if (MP == 32)
            hipLaunchKernelGGL(k_masks_plrnn<32>, dim3(grid), dim3(256), 0, st, a.alpha, a.N, a.x, a.z0, z, masks, active, a.B, a.T, a.M, a.tw);
        else
            hipLaunchKernelGGL(k_masks_plrnn<64>, dim3(grid), dim3(256), 0, st, a.alpha, a.N, a.x, a.z0, z, masks, active, a.B, a.T, a.M, a.tw);
        DEER_LAUNCH_CHECK("k_masks_plrnn");
        return DEER_OK;
    }
    if (a.tw > 0) return invalid_arg("the residual kernel takes no latent warm-up");
    const long groups = ((long)a.B * a.T + (64 / MP) - 1) / (64 / MP);
    const long passes = J ? groups : (groups + 3) / 4;
    const int grid = (int)(passes < 8192 ? passes : 8192);
    KTimer kt("k_resjac_plrnn", st);
#define RJ(MPV, DJ)                                                                                                 \
    hipLaunchKernelGGL((k_resjac_plrnn<MPV, DJ>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x, a.z0, \
                       z, F, r, J, masks, active, a.B, a.T, a.M)
    if (J) {
        if (MP == 16) RJ(16, true); else if (MP == 32) RJ(32, true); else RJ(64, true);
    } else {
        if (MP == 16) RJ(16, false); else if (MP == 32) RJ(32, false); else RJ(64, false);
    }
#undef RJ
    DEER_LAUNCH_CHECK("k_resjac_plrnn");
    return DEER_OK;
}

int launch_chunk_product_plrnn(const PlrnnArgs &a, bool rev, const uint32_t *masks, const float *rhs, const float *z,
                               float seed_scale, float *P, float *v, const int *active, int C, int ncs,
                               hipStream_t st) {
    const int MP = padded(a.M);
    const int nch = a.B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt("k_chunk_product_plrnn", st);
#define CP(MPV, R, WUV)                                                                                              \
    hipLaunchKernelGGL((k_chunk_product_plrnn<MPV, R, WUV>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N,    \
                       masks, rhs, z, a.x, seed_scale, P, v, active, a.B, a.T, a.M, C, ncs, a.tw)
#define CPW(MPV, R) \
    if (a.tw > 0) CP(MPV, R, true); else CP(MPV, R, false);
    if (!rev) {
        if (MP == 16) { CPW(16, false) } else if (MP == 32) { CPW(32, false) } else { CPW(64, false) }
    } else {
        if (MP == 16) { CPW(16, true) } else if (MP == 32) { CPW(32, true) } else { CPW(64, true) }
    }
#undef CPW
#undef CP
    DEER_LAUNCH_CHECK("k_chunk_product_plrnn");
    return DEER_OK;
}

int launch_newton_product_plrnn(const PlrnnArgs &a, const float *z, const float *zalt, const int *zsel, float *r,
                                uint32_t *masks, float *P, float *v, const int *active, const float *gamma, int C,
                                int ncs, int wmaps, float *gmap, uint32_t *mark, uint32_t pass_no, hipStream_t st) {
    const int MP = padded(a.M);
    const int nch = a.B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt("k_newton_product_plrnn", st);
    if (wmaps == 2 && (MP != 16 || ncs % 32 || !gmap))
        return invalid_arg("group maps need M <= 16, a chunk count divisible by 32 and their buffer");
#define NP(MPV)                                                                                                    \
    if (a.tw > 0)                                                                                                  \
        hipLaunchKernelGGL((k_newton_product_plrnn<MPV, true>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, \
                           a.N, a.x, a.z0, z, zalt, zsel, r, masks, P, v, active, gamma, a.B, a.T, a.M, C, ncs, a.tw); \
    else                                                                                                           \
        hipLaunchKernelGGL((k_newton_product_plrnn<MPV, false>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, \
                           a.N, a.x, a.z0, z, zalt, zsel, r, masks, P, v, active, gamma, a.B, a.T, a.M, C, ncs, 0)
    if (wmaps && (MP != 16 || ncs % 4))
        return invalid_arg("composed wave maps need M <= 16 and a chunk count divisible by 4");
    if (mark && MP != 16) return invalid_arg("pass marks are written by the M <= 16 forward pass only");
    if (MP == 64 && (a.N == 0 || a.N == a.M)) {   // uniform forcing factor: W-in-LDS kernel
        if (a.tw > 0)
            hipLaunchKernelGGL(k_newton_product_plrnn64u<true>, dim3(nch), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, a.N,
                               a.x, a.z0, z, zalt, zsel, r, masks, P, v, active, gamma, a.B, a.T, a.M, C, ncs, a.tw);
        else
            hipLaunchKernelGGL(k_newton_product_plrnn64u<false>, dim3(nch), dim3(64), 0, st, a.A, a.W, a.h, a.alpha,
                               a.N, a.x, a.z0, z, zalt, zsel, r, masks, P, v, active, gamma, a.B, a.T, a.M, C, ncs, 0);
    } else if (MP == 16) {
#define NP16(TBV, WPBV)                                                                                                \
    hipLaunchKernelGGL((k_newton_product_plrnn16<TBV, WPBV, WUV>), dim3(grid / WPBV), dim3(64 * WPBV), 0, st, a.A, a.W, \
                       a.h, a.alpha, a.N, a.x, a.z0, z, zalt, zsel, P, v, active, gamma, a.B, a.T, a.M, C, ncs, wmaps, \
                       gmap, mark, pass_no, a.tw)
#define NP16W(TBV, WPBV)            \
    if (a.tw > 0) {                 \
        constexpr bool WUV = true;  \
        NP16(TBV, WPBV);            \
    } else {                        \
        constexpr bool WUV = false; \
        NP16(TBV, WPBV);            \
    }
        if (wmaps == 2) {
            if (C % 32) { NP16W(16, 8) } else { NP16W(32, 8) }
        } else {
            if (C % 32) { NP16W(16, 1) } else { NP16W(32, 1) }
        }
#undef NP16W
#undef NP16
    } else if (MP == 32) {
        NP(32);
    } else {
        NP(64);
    }
#undef NP
    DEER_LAUNCH_CHECK("k_newton_product_plrnn");
    return DEER_OK;
}

int launch_newton_pass16(const PlrnnArgs &a, float *z, float *zalt, const float *Pin, const float *vin,
                         const float *gin, float *Pout, float *vout, float *gout, int C, int ncs, const FusedCtl &fc,
                         uint32_t *mark, uint32_t pass_no, hipStream_t st) {
    if (a.M > 16 || ncs % 32 || C % 16 || (long)C * ncs != a.T || !fc.seq || !fc.nd.pv || !Pin || !vin || !gin ||
        !Pout || !vout || !gout)
        return invalid_arg("fused Newton passes need M <= 16, 32 | chunks, 16 | C, T = C chunks, the control and "
                           "two aggregate buffers");
    KTimer kt("k_newton_pass16", st);
    const int grid = a.B * ncs / 32;
#define NPS(TBV)                                                                                                  \
    hipLaunchKernelGGL((k_newton_pass16<TBV, WUV>), dim3(grid), dim3(512), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x,  \
                       a.z0, z, zalt, a.T, a.M, C, ncs, Pin, vin, gin, Pout, vout, gout, fc, mark, pass_no, a.tw)
    if (a.tw > 0) {
        constexpr bool WUV = true;
        if (C % 32) NPS(16); else NPS(32);
    } else {
        constexpr bool WUV = false;
        if (C % 32) NPS(16); else NPS(32);
    }
#undef NPS
    DEER_LAUNCH_CHECK("k_newton_pass16");
    return DEER_OK;
}

// two-level carry for chunk sequences at least this long
static int carry_group_size(int MP, int ncs) {
    if (MP == 128) {
        // a group step (a 128 x 128 x 128 product on one CU) costs about six walk steps
        if (ncs < 48) return 0;
        int G = 4;
        while (8 * G * G < ncs) G <<= 1;
        return G;
    }
    if (ncs < 96) return 0;
    int G = 8;
    while (2 * G * G < ncs) G <<= 1;   // a group step costs about twice a walk step
    return G;
}

size_t carry_ws_floats(int MP, int B, int ncs) {
    const int G = carry_group_size(MP, ncs);
    if (!G) return 0;
    const size_t ng = (size_t)(ncs + G - 1) / G;
    return (size_t)B * ng * ((size_t)MP * MP + 2 * MP);
}

int launch_carry(int MP, bool rev, const float *P, const float *v, float *carry_in, const int *active,
                 uint32_t *norm_bits, int B, int ncs, float *gws, hipStream_t st) {
    if (MP == 128) {
        if (norm_bits) return invalid_arg("width-128 carries take no norms");
        return launch_carry_big(rev, P, v, carry_in, active, B, ncs, gws ? carry_group_size(MP, ncs) : 0, gws, st);
    }
    KTimer kt("k_carry", st);
    const int G = gws ? carry_group_size(MP, ncs) : 0;
#define CA(MPV, R, PP, VV, CI, NB, NC, GG, ST, GRID) \
    hipLaunchKernelGGL((k_carry<MPV, R>), dim3(GRID), dim3(MPV), 0, st, PP, VV, CI, active, NB, B, NC, GG, ST)
#define CG(MPV, R, GRID) \
    hipLaunchKernelGGL((k_carry_group<MPV, R>), dim3(GRID), dim3(256), 0, st, P, v, gq, gu, active, ncs, G)
    if (!G) {
        if (MP == 16) {
            if (rev)
                hipLaunchKernelGGL(k_carry16<true>, dim3(B), dim3(64), 0, st, P, v, carry_in, active, norm_bits, B, ncs, ncs, nullptr);
            else
                hipLaunchKernelGGL(k_carry16<false>, dim3(B), dim3(64), 0, st, P, v, carry_in, active, norm_bits, B, ncs, ncs, nullptr);
        } else if (!rev) {
            if (MP == 16) CA(16, false, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
            else if (MP == 32) CA(32, false, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
            else CA(64, false, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
        } else {
            if (MP == 16) CA(16, true, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
            else if (MP == 32) CA(32, true, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
            else CA(64, true, P, v, carry_in, norm_bits, ncs, ncs, nullptr, B);
        }
    } else {
        const int ng = (ncs + G - 1) / G;
        float *gq = gws;
        float *gu = gq + (size_t)B * ng * MP * MP;
        float *gc = gu + (size_t)B * ng * MP;
        const int grid = B * ng;
#define CG3(MPV)                                                             \
    {                                                                        \
        if (rev) CG(MPV, true, grid); else CG(MPV, false, grid);             \
        CA(MPV, false, gq, gu, gc, nullptr, ng, ng, nullptr, B);             \
        if (rev) CA(MPV, true, P, v, carry_in, norm_bits, ncs, G, gc, grid); \
        else CA(MPV, false, P, v, carry_in, norm_bits, ncs, G, gc, grid);    \
    }
        if (MP == 16) {
            if (rev) hipLaunchKernelGGL(k_carry_group16<true>, dim3(grid), dim3(64), 0, st, P, v, gq, gu, active, ncs, G);
            else hipLaunchKernelGGL(k_carry_group16<false>, dim3(grid), dim3(64), 0, st, P, v, gq, gu, active, ncs, G);
            hipLaunchKernelGGL(k_carry16<false>, dim3(B), dim3(64), 0, st, gq, gu, gc, active, nullptr, B, ng, ng, nullptr);
            if (rev)
                hipLaunchKernelGGL(k_carry16<true>, dim3(grid), dim3(64), 0, st, P, v, carry_in, active, norm_bits, B, ncs, G, gc);
            else
                hipLaunchKernelGGL(k_carry16<false>, dim3(grid), dim3(64), 0, st, P, v, carry_in, active, norm_bits, B, ncs, G, gc);
        } else if (MP == 32) CG3(32) else CG3(64)
#undef CG3
    }
#undef CG
#undef CA
    DEER_LAUNCH_CHECK("k_carry");
    return DEER_OK;
}

int launch_carry_walk16(bool rev, const float *P, const float *v, float *carry, const int *active, int B, int ncs,
                        hipStream_t st) {
    if (ncs % 4) return invalid_arg("wave-map walk needs a chunk count divisible by 4");
    KTimer kt("k_carry", st);
    if (rev) hipLaunchKernelGGL(k_carry_walk16<true>, dim3(B), dim3(WALK_NWV * 64), 0, st, P, v, carry, active, ncs);
    else hipLaunchKernelGGL(k_carry_walk16<false>, dim3(B), dim3(WALK_NWV * 64), 0, st, P, v, carry, active, ncs);
    DEER_LAUNCH_CHECK("k_carry_walk16");
    return DEER_OK;
}

// 16 < M <= 64: the forward fix-up on the matrix cores unless DEER_FIX_MFMA=0
static bool fixup_mfma() {
    const char *e = getenv("DEER_FIX_MFMA");
    return !e || atoi(e) != 0;
}

int launch_fixup_fwd_plrnn(const PlrnnArgs &a, const uint32_t *masks, const float *r, const float *carry_in,
                           float *z, float *zalt, const int *zsel, uint32_t *chain_bits, const int *active,
                           const float *gamma, int C, int ncs, const float *Pm, const float *vm,
                           const float *gmap, const FusedCtl *fc, hipStream_t st) {
    const int MP = padded(a.M);
    const int nch = a.B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt("k_fixup_fwd_plrnn", st);
#define FX(MPV)                                                                                                        \
    if (a.tw > 0)                                                                                                      \
        hipLaunchKernelGGL((k_fixup_fwd_plrnn<MPV, true>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N, masks, r, \
                           carry_in, z, zalt, zsel, chain_bits, active, gamma, a.B, a.T, a.M, C, ncs, a.tw);        \
    else                                                                                                               \
        hipLaunchKernelGGL((k_fixup_fwd_plrnn<MPV, false>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N, masks, \
                           r, carry_in, z, zalt, zsel, chain_bits, active, gamma, a.B, a.T, a.M, C, ncs, 0)
#define FX16(TBV)                                                                                                 \
    hipLaunchKernelGGL((k_fixup_fwd_plrnn16<TBV, WUV>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x,  \
                       a.z0, carry_in, z, zalt, zsel, chain_bits, active, gamma, a.B, a.T, a.M, C, ncs, Pm, vm, gmap, \
                       fcv, a.tw)
    if (gmap && (!Pm || ncs % 32)) return invalid_arg("group maps need the wave maps and 32 | chunk count");
    if (Pm && (MP != 16 || ncs % 4))
        return invalid_arg("composed wave maps need M <= 16 and a chunk count divisible by 4");
    if (fc && MP != 16) return invalid_arg("the fused pass-end control needs M <= 16");
    FusedCtl fcv{};
    if (fc) fcv = *fc;
    if (MP == 16) {
        if (a.tw > 0) {
            constexpr bool WUV = true;
            if (C % 32) FX16(16); else FX16(32);
        } else {
            constexpr bool WUV = false;
            if (C % 32) FX16(16); else FX16(32);
        }
    } else if (fixup_mfma()) {
        const int gridm = (nch + 15) / 16;
#define FXM(MPV, VV)                                                                                                  \
    if (a.tw > 0)                                                                                                     \
        hipLaunchKernelGGL((k_fixup_fwd_plrnn_mf<MPV, VV, true>), dim3(gridm), dim3(MPV * 4), 0, st, a.A, a.W, a.alpha, \
                           a.N, masks, r, carry_in, z, zalt, zsel, chain_bits, active, gamma, a.B, a.T, a.M, C, ncs,  \
                           a.tw);                                                                                     \
    else                                                                                                              \
        hipLaunchKernelGGL((k_fixup_fwd_plrnn_mf<MPV, VV, false>), dim3(gridm), dim3(MPV * 4), 0, st, a.A, a.W,       \
                           a.alpha, a.N, masks, r, carry_in, z, zalt, zsel, chain_bits, active, gamma, a.B, a.T, a.M, \
                           C, ncs, 0)
        const bool v4 = (a.M & 3) == 0;
        if (MP == 32) {
            if (v4) { FXM(32, true); } else { FXM(32, false); }
        } else {
            if (v4) { FXM(64, true); } else { FXM(64, false); }
        }
#undef FXM
    } else if (MP == 32) {
        FX(32);
    } else {
        FX(64);
    }
#undef FX16
#undef FX
    DEER_LAUNCH_CHECK("k_fixup_fwd_plrnn");
    return DEER_OK;
}

int launch_fixup_rev_plrnn(const PlrnnArgs &a, const uint32_t *masks, const float *g, float seed_scale, const float *z,
                           const float *carry_in, float *lam, float *gpart, int C, int ncs, hipStream_t st) {
    const int MP = padded(a.M);
    const int nch = a.B * ncs;
    const int grid = (nch + (64 / MP) - 1) / (64 / MP);
    KTimer kt("k_fixup_rev_plrnn", st);
#define FR(MPV)                                                                                                      \
    if (a.tw > 0)                                                                                                    \
        hipLaunchKernelGGL((k_fixup_rev_plrnn<MPV, true>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N, masks, \
                           g, seed_scale, a.x, a.z0, z, carry_in, lam, gpart, a.B, a.T, a.M, C, ncs, a.tw);         \
    else                                                                                                             \
        hipLaunchKernelGGL((k_fixup_rev_plrnn<MPV, false>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N,     \
                           masks, g, seed_scale, a.x, a.z0, z, carry_in, lam, gpart, a.B, a.T, a.M, C, ncs, 0)
    if (MP == 16) {
        FR(16);
    } else if (MP == 32) {
        FR(32);
    } else {
        FR(64);
    }
#undef FR
    DEER_LAUNCH_CHECK("k_fixup_rev_plrnn");
    return DEER_OK;
}

int launch_adjoint_plrnn16(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *P, float *v,
                           float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st) {
    if (padded(a.M) != 16) return invalid_arg("the register-tiled adjoint needs M <= 16");
    const int nch = a.B * ncs, grid = (nch + 3) / 4;
    const bool wm = ncs % 4 == 0;
    {
        KTimer kt("k_chunk_product_plrnn", st);
#define CPR(TBV)                                                                                                     \
    hipLaunchKernelGGL((k_chunk_product_plrnn16_rev<TBV, WUV>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N, \
                       g, z, a.x, seed_scale, P, v, a.B, a.T, a.M, C, ncs, (int)wm, a.tw)
        if (a.tw > 0) {   // 16-step tiles: the warm-up variant's registers fit two waves per SIMD
            constexpr bool WUV = true;
            CPR(16);
        } else {
            constexpr bool WUV = false;
            if (C % 32) CPR(16); else CPR(32);
        }
#undef CPR
        DEER_LAUNCH_CHECK("k_chunk_product_plrnn16_rev");
    }
    int rc;
    if (wm) rc = launch_carry_walk16(true, P, v, carry, nullptr, a.B, ncs, st);
    else rc = launch_carry(16, true, P, v, carry, nullptr, nullptr, a.B, ncs, nullptr, st);
    if (rc) return rc;
    {
        KTimer kt("k_fixup_rev_plrnn", st);
#define FRV(TBV)                                                                                                   \
    hipLaunchKernelGGL((k_fixup_rev_plrnn16<TBV, WUV>), dim3(grid), dim3(64), 0, st, a.A, a.W, a.alpha, a.N, g,       \
                       seed_scale, a.x, a.z0, z, carry, wm ? P : nullptr, wm ? v : nullptr, lam, gpart, a.B, a.T, a.M, C, \
                       ncs, a.tw)
        if (a.tw > 0) {
            constexpr bool WUV = true;
            FRV(16);
        } else {
            constexpr bool WUV = false;
            if (C % 32) FRV(16); else FRV(32);
        }
#undef FRV
        DEER_LAUNCH_CHECK("k_fixup_rev_plrnn16");
    }
    return DEER_OK;
}

int launch_reduce_gpart(const float *gpart, int nchains, int MP, int M, float *dA, float *dW, float *dh,
                        double *part2, hipStream_t st) {
    const int n = MP * (MP + 2);
    {
        KTimer _kt("k_reduce_gpart", st);
        hipLaunchKernelGGL(k_reduce_gpart1, dim3(GP_SLICES, (n + 63) / 64), dim3(256), 0, st, gpart, nchains, n, part2);
        hipLaunchKernelGGL(k_reduce_gpart2, dim3((n + 255) / 256), dim3(256), 0, st, (const double *)part2, MP, M, dA,
                           dW, dh);
    }
    DEER_LAUNCH_CHECK("k_reduce_gpart");
    return DEER_OK;
}

int padded_dim(int M) { return padded(M); }

}  // namespace deer
