// Shallow PLRNN Newton update without a stored Jacobian (eq. shplrnn_nonlinear with V = W2,
// b = h2; eq. GTF_DEER_update).  The forced Jacobian of step t,
//   J~_t = gamma (diag(A p) + W1 diag(m_t) W2 diag(p)),   m_t = (W2 z~_{t-1} + h2 > 0),
// is never written to HBM: the residual kernel leaves the hidden masks m_t (L bits per step),
// and the two kernels here rebuild what they need of J~_t from them and from W1, W2.
//
//   k_chunk_product_shfused  per chunk, J~_t^T formed on the matrix cores (K = L, the masks
//        applied to the W1 operand) lands in exactly the register layout of an A operand of
//        J~_t, so the composition P <- J~_t P and the local solution u <- J~_t u + s r_t follow
//        at once, as in the stored-Jacobian chunk product.  A wave owns one chunk and forms
//        the Jacobians of NT consecutive steps per pass over the W1 / W2 tiles in LDS.
//   k_fixup_shjvp            the chunk re-run from its carry with J~_t applied as a
//        Jacobian-vector product, Delta_t = gamma (A p Delta + W1 (m_t (W2 (p Delta)))) + s r_t.
//        A block runs 16 chains as the 16 columns of two matrix-core products per step; its 4
//        waves split the hidden units, hold their slices of W2 diag(p) and W1 as A fragments in
//        registers for the whole chunk, and sum their partial W1 products through LDS.
// Per step this replaces 4 M^2 bytes written and read twice by 4 L / 8 bytes of masks.
#include "common.h"
#include "launch.h"
#include "newton_ctl.h"

namespace deer {

__device__ __forceinline__ float pf_at(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

static int shf_LP(int L) { return (L + 15) / 16 * 16; }

size_t shfused_product_lds(int M, int L) {
    return (size_t)2 * padded_dim(M) * (shf_LP(L) + 4) * sizeof(float);
}

// l tiles per wave of the fix-up (4 waves share the (L + 15) / 16 tiles)
static int shf_nlw(int L) {
    const int nlt = (L + 15) / 16;
    const int per = (nlt + 3) / 4;
    return per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : per <= 8 ? 8 : 0;
}

size_t shf_resjac_lds(int M, int L);

bool shfused_supported(int M, int L) {
    const int MP = padded_dim(M);
    if (MP > 64 || L <= 0) return false;
    // two blocks per CU
    if (shfused_product_lds(M, L) > 80 * 1024 || shf_resjac_lds(M, L) > 80 * 1024) return false;
    const int nlw = shf_nlw(L);
    // fix-up A fragments in registers: NLW * (MP / 4) + (MP / 16) * 4 NLW floats per lane
    return nlw > 0 && nlw * (MP / 4 + MP / 4) <= 64;
}

// ---------------------------------------------------------------------------------------
// Jacobian formation shared by the two chunk products.  LDS: w2t [MP][LQ] = (W2 diag(p))^T
// (row i, column l) and w1s [MP][LQ] = W1 (row j, column l), LQ = LP + 4 (the rows read by a
// 16-lane group fall on different banks).
// jt tile (I, Jt) of step nt: lane (g, c) element r = J^T[16I + 4g + r][16Jt + c]
//   = J[16Jt + c][16I + 4g + r]   (J = W1 diag(m) W2 diag(p), without the diagonal),
// which is the A fragment of row tile Jt, k-step 4I + r of a product J X (lane (g, c) of an A
// fragment holds J[16I' + c][16j + 4g + q]).
// ---------------------------------------------------------------------------------------
template <int MP>
__device__ __forceinline__ void shf_stage_weights(const ShArgs &a, float *w2t, float *w1s, int LQ) {
    const int M = a.M, L = a.L, N = a.N;
    for (int e = threadIdx.x; e < MP * LQ; e += 256) {
        const int i = e / LQ, l = e % LQ;
        const bool ok = i < M && l < L;
        w2t[e] = ok ? a.W2[(size_t)l * M + i] * pf_at(i, N, a.alpha) : 0.f;
        w1s[e] = ok ? a.W1[(size_t)i * L + l] : 0.f;
    }
}

// jt of the steps whose mask rows are row_first + nt, nt < nvalid (wave-uniform, <= NT)
template <int MP, int NT>
__device__ __forceinline__ void shf_form(const float *w2t, const float *w1s, int LQ, int njl,
                                         const uint32_t *__restrict__ masks, int LW, size_t row_first, int nvalid,
                                         int g, int c, v4f (&jt)[NT][MP / 16][MP / 16]) {
    constexpr int NI = MP / 16;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int Jt = 0; Jt < NI; ++Jt) jt[nt][I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
    // mask words: one per pair of 16-unit k tiles, loaded a pair ahead
    uint32_t mw[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) mw[nt] = nt < nvalid ? masks[(row_first + nt) * LW] : 0u;
    // LDS operands of k tile j, read one tile ahead of their matrix-core instructions
    float4 av[NI], bv[NI];
    auto lds_ops = [&](int j, float4 (&ao)[NI], float4 (&bo)[NI]) {
#pragma unroll
        for (int I = 0; I < NI; ++I) ao[I] = *reinterpret_cast<const float4 *>(w2t + (16 * I + c) * LQ + 16 * j + 4 * g);
#pragma unroll
        for (int Jt = 0; Jt < NI; ++Jt)
            bo[Jt] = *reinterpret_cast<const float4 *>(w1s + (16 * Jt + c) * LQ + 16 * j + 4 * g);
    };
    lds_ops(0, av, bv);
    for (int jp = 0; jp < njl; jp += 2) {
        uint32_t mc[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            mc[nt] = mw[nt];
            const int wn = (jp >> 1) + 1;
            mw[nt] = (nt < nvalid && wn < LW) ? masks[(row_first + nt) * LW + wn] : 0u;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int j = jp + h;
            if (j >= njl) break;
            float4 an[NI], bn[NI];
            lds_ops(j + 1 < njl ? j + 1 : j, an, bn);
            const int sh = 16 * h + 4 * g;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                if (nt >= nvalid) continue;
                const uint32_t w = mc[nt];
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt) {
                    const float b0 = select_bit(w, sh + 0, bv[Jt].x), b1 = select_bit(w, sh + 1, bv[Jt].y);
                    const float b2 = select_bit(w, sh + 2, bv[Jt].z), b3 = select_bit(w, sh + 3, bv[Jt].w);
#pragma unroll
                    for (int I = 0; I < NI; ++I) {
                        v4f t = jt[nt][I][Jt];
                        t = mfma16x16x4(av[I].x, b0, t);
                        t = mfma16x16x4(av[I].y, b1, t);
                        t = mfma16x16x4(av[I].z, b2, t);
                        t = mfma16x16x4(av[I].w, b3, t);
                        jt[nt][I][Jt] = t;
                    }
                }
            }
#pragma unroll
            for (int I = 0; I < NI; ++I) {
                av[I] = an[I];
                bv[I] = bn[I];
            }
        }
    }
}

// A fragments of J~ = gm (J + diag(A p)) from one step's jt: row tile I, k-step s = 4j + q
// holds J~[16I + c][16j + 4g + q]; dg[I] = A_i p_i of row i = 16I + c
template <int MP>
__device__ __forceinline__ void shf_afrag(const v4f (&jt)[MP / 16][MP / 16], const float (&dg)[MP / 16], float gm,
                                          int g, int c, float (&ac)[MP / 16][MP / 4]) {
    constexpr int NI = MP / 16;
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float v = jt[j][I][q];
                if (I == j && c == 4 * g + q) v = v + dg[I];
                ac[I][4 * j + q] = gm * v;
            }
}

// a latent warm-up step's P_1 (section "Latent state warm-up"): the observed latents' columns of
// J~ (k-steps 16 j + 4 g + q < N) dropped from its A fragments
template <int MP>
__device__ __forceinline__ void shf_drop_observed(float (&ac)[MP / 16][MP / 4], int N, int g) {
    constexpr int NI = MP / 16;
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (16 * j + 4 * g + q < N) ac[I][4 * j + q] = 0.f;
}

// ---------------------------------------------------------------------------------------
// forward chunk product: per chain the B operand is [P | u] (P's MP/16 column tiles plus one
// whose column 0 is u), P <- J~_t P and u <- J~_t u + rhs_sign r_t, with P = I and u = 0 at
// the chunk start (the stored-Jacobian kernel's contract: P and the local solution v per chain).
// ---------------------------------------------------------------------------------------
template <int MP, int NT>
__global__ __launch_bounds__(256) void k_chunk_product_shfused(const ShArgs a, const uint32_t *__restrict__ masks,
                                                               const float *__restrict__ rhs, float rhs_sign,
                                                               const float *__restrict__ gamma,
                                                               float *__restrict__ Pout, float *__restrict__ vout,
                                                               const int *__restrict__ active, int C, int ncs,
                                                               int LP) {
    constexpr int NI = MP / 16, NS = MP / 4, PT = MP / 16;
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, N = a.N, LQ = LP + 4;
    float *w2t = smem;
    float *w1s = smem + MP * LQ;
    shf_stage_weights<MP>(a, w2t, w1s, LQ);
    __syncthreads();
    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    const int nchains = a.B * ncs;
    const int id = blockIdx.x * 4 + wv;
    const bool exists = id < nchains;
    const int b = exists ? id / ncs : 0, cc = exists ? id % ncs : 0;
    const bool ok = exists && (!active || active[b]);
    const int s0 = cc * C;
    const int len = __builtin_amdgcn_readfirstlane(ok ? max(min(s0 + C, T) - s0, 0) : 0);
    const float gm = gamma ? gamma[b] : 1.f;
    float dg[NI];
#pragma unroll
    for (int I = 0; I < NI; ++I) {
        const int row = 16 * I + c;
        dg[I] = row < M ? a.A[row] * pf_at(row, N, a.alpha) : 0.f;
    }
    v4f acc[PT + 1][NI];
#pragma unroll
    for (int tt = 0; tt <= PT; ++tt)
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                acc[tt][I][r] = (tt < PT && 16 * I + 4 * g + r == 16 * tt + c) ? 1.f : 0.f;
    const size_t row0 = (size_t)b * T + s0;
    const int njl = LP / 16;
    for (int t0 = 0; t0 < len; t0 += NT) {
        const int nv = min(NT, len - t0);
        // right-hand sides of the NT steps (lanes of column 0), loaded before the formation
        float rc[NT][NI][4];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = 16 * I + 4 * g + r;
                    rc[nt][I][r] = (nt < nv && c == 0 && row < M) ? rhs[(row0 + t0 + nt) * M + row] : 0.f;
                }
        v4f jt[NT][NI][NI];
        shf_form<MP, NT>(w2t, w1s, LQ, njl, masks, LW, row0 + t0, nv, g, c, jt);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (nt >= nv) break;
            float ac[NI][NS];
            shf_afrag<MP>(jt[nt], dg, gm, g, c, ac);
            if (a.tw > 0 && s0 + t0 + nt <= a.tw) shf_drop_observed<MP>(ac, N, g);
#pragma unroll
            for (int tt = 0; tt <= PT; ++tt) {
                float Bop[NS];
#pragma unroll
                for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) Bop[4 * j + q] = acc[tt][j][q];
#pragma unroll
                for (int I = 0; I < NI; ++I) {
                    v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k = 0; k < NS; ++k) s = mfma16x16x4(ac[I][k], Bop[k], s);
                    acc[tt][I] = s;
                }
            }
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[PT][I][r] = fmaf(rhs_sign, rc[nt][I][r], acc[PT][I][r]);
        }
    }
    if (!exists) return;
    if (len > 0) {
        float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
        for (int tt = 0; tt < PT; ++tt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) P[(16 * I + 4 * g + r) * MP + 16 * tt + c] = acc[tt][I][r];
    }
    if (c == 0) {
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) vout[(size_t)id * MP + 16 * I + 4 * g + r] = acc[PT][I][r];
    }
}

// ---------------------------------------------------------------------------------------
// reverse chunk product (adjoint, eq. backward_recursion: y_k = J~_{k+1}^T y_{k+1} + s b_k).
// Chunk [s0, s1) stores the stored-Jacobian kernel's pair: Q = J~_{hi-1} ... J~_{s0+1}
// (hi = min(s1 + 1, T); the carry pass applies Q^T) and the local solution from a zero carry,
//   v = y_{s0} = sum_{k = s0}^{s1 - 1} Q_k^T (s b_k),   Q_k = J~_k ... J~_{s0+1},  Q_{s0} = I,
// which the forward sweep that builds Q accumulates on the way: at step k first v += Q^T s b_k
// (each lane adds the products of its rows of a column; the 4 lane groups' sums are added at
// the end), then Q <- J~_{k+1} Q.  Undamped (the adjoint is taken at the solution).
// ---------------------------------------------------------------------------------------
template <int MP, int NT>
__global__ __launch_bounds__(256) void k_chunk_product_shfused_rev(const ShArgs a, const uint32_t *__restrict__ masks,
                                                                   const float *__restrict__ rhs, float rhs_sign,
                                                                   float *__restrict__ Pout, float *__restrict__ vout,
                                                                   int C, int ncs, int LP) {
    constexpr int NI = MP / 16, NS = MP / 4, PT = MP / 16;
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, N = a.N, LQ = LP + 4;
    float *w2t = smem;
    float *w1s = smem + MP * LQ;
    shf_stage_weights<MP>(a, w2t, w1s, LQ);
    __syncthreads();
    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    const int nchains = a.B * ncs;
    const int id = blockIdx.x * 4 + wv;
    const bool exists = id < nchains;
    const int b = exists ? id / ncs : 0, cc = exists ? id % ncs : 0;
    const int s0 = cc * C;
    const int len = __builtin_amdgcn_readfirstlane(exists ? max(min(s0 + C, T) - s0, 0) : 0);
    float dg[NI];
#pragma unroll
    for (int I = 0; I < NI; ++I) {
        const int row = 16 * I + c;
        dg[I] = row < M ? a.A[row] * pf_at(row, N, a.alpha) : 0.f;
    }
    v4f acc[PT][NI];
#pragma unroll
    for (int tt = 0; tt < PT; ++tt)
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[tt][I][r] = (16 * I + 4 * g + r == 16 * tt + c) ? 1.f : 0.f;
    float vc[PT];   // this lane group's part of element 16 tt + c of the local solution
#pragma unroll
    for (int tt = 0; tt < PT; ++tt) vc[tt] = 0.f;
    const size_t row0 = (size_t)b * T + s0;
    const int njl = LP / 16;
    for (int t0 = 0; t0 < len; t0 += NT) {
        const int nv = min(NT, len - t0);
        // J~_{k+1} exists for k + 1 < T
        const int nj = max(0, min(nv, T - 1 - (s0 + t0)));
        float bk[NT][NI][4];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = 16 * I + 4 * g + r;
                    bk[nt][I][r] = (nt < nv && row < M) ? rhs_sign * rhs[(row0 + t0 + nt) * M + row] : 0.f;
                }
        v4f jt[NT][NI][NI];
        shf_form<MP, NT>(w2t, w1s, LQ, njl, masks, LW, row0 + t0 + 1, nj, g, c, jt);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (nt >= nv) break;
#pragma unroll
            for (int tt = 0; tt < PT; ++tt) {
#pragma unroll
                for (int I = 0; I < NI; ++I)
#pragma unroll
                    for (int r = 0; r < 4; ++r) vc[tt] = fmaf(acc[tt][I][r], bk[nt][I][r], vc[tt]);
            }
            if (nt >= nj) continue;
            float ac[NI][NS];
            shf_afrag<MP>(jt[nt], dg, 1.f, g, c, ac);
            if (a.tw > 0 && s0 + t0 + nt + 1 <= a.tw) shf_drop_observed<MP>(ac, N, g);   // J~_{k+1}
#pragma unroll
            for (int tt = 0; tt < PT; ++tt) {
                float Bop[NS];
#pragma unroll
                for (int j = 0; j < NS / 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) Bop[4 * j + q] = acc[tt][j][q];
#pragma unroll
                for (int I = 0; I < NI; ++I) {
                    v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k = 0; k < NS; ++k) s = mfma16x16x4(ac[I][k], Bop[k], s);
                    acc[tt][I] = s;
                }
            }
        }
    }
    if (!exists) return;
    if (len > 0) {
        float *P = Pout + (size_t)id * MP * MP;
#pragma unroll
        for (int tt = 0; tt < PT; ++tt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) P[(16 * I + 4 * g + r) * MP + 16 * tt + c] = acc[tt][I][r];
    }
    // the lane groups' partial sums of each column
#pragma unroll
    for (int tt = 0; tt < PT; ++tt) {
        vc[tt] += __shfl_xor(vc[tt], 16, 64);
        vc[tt] += __shfl_xor(vc[tt], 32, 64);
    }
    if (g == 0) {
#pragma unroll
        for (int tt = 0; tt < PT; ++tt) vout[(size_t)id * MP + 16 * tt + c] = vc[tt];
    }
}

// ---------------------------------------------------------------------------------------
// fix-ups.  Block = 16 chains (column c = lane & 15) x 4 waves; wave w owns the l tiles
// lt = NLW w + k.  Per step, with y tiles dl[I] (lane (g, c) element r = y[16I + 4g + r] of
// chain c, replicated in all 4 waves):
//   forward (Newton, REV false), J~_t y at step k = s0 + t, masks of step k:
//     u[k] = (W2 diag(p))[tile lt, :] y,  u *= m,  p2[I] = W1[tile I, wave's tiles] u
//     next = gamma (p2 + A p y) - r_k; z_k += next, per-chain max |Delta| and max |z|
//   reverse (adjoint, REV true), J~_{k+1}^T y at step k = s1 - 1 - t, masks of step k + 1:
//     u[k] = W1^T[tile lt, :] y,  u *= m,  p2[I] = (W2 diag(p))^T[tile I, wave's tiles] u
//     next = (p2 + A p y) + s g_k  (no J term when k + 1 = T); y_k written
// A = the first factor's rows as A fragments, B = y or u in the k-permuted accumulator layout.
// The waves' contributions (wave 0 adds the diagonal and the right-hand side) are summed in
// LDS in a fixed order, so every wave holds the same next y.
// ---------------------------------------------------------------------------------------
template <int MP, int NLW, bool REV>
__global__ __launch_bounds__(256) void k_fixup_shjvp(const ShArgs a, const uint32_t *__restrict__ masks,
                                                     const float *__restrict__ rhs, float rhs_sign,
                                                     const float *__restrict__ gamma,
                                                     const float *__restrict__ carry_in, float *zbuf, float *outbuf,
                                                     const int *__restrict__ zsel, uint32_t *__restrict__ chain_bits,
                                                     const int *__restrict__ active, int C, int ncs, FusedCtl fc) {
    constexpr int NI = MP / 16, NS = MP / 4;
    __shared__ v4f red[2][4][NI][64];
    const int tid = threadIdx.x, wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4,
              c = lane & 15;
    const int M = a.M, L = a.L, T = a.T, N = a.N;
    const int LW = (L + 31) / 32, nlt = (L + 15) / 16;
    // a1: rows l = 16 lt + c, k = i = 16 j + 4 g + q;  a2: rows i = 16 I + c, k = l = 16 lt + 4 g + q
    float a1[NLW][NS], a2[NI][4 * NLW];
#pragma unroll
    for (int k = 0; k < NLW; ++k) {
        const int lt = wv * NLW + k, l = 16 * lt + c;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int i = 16 * (s / 4) + 4 * g + (s % 4);
            const bool e = lt < nlt && l < L && i < M;
            a1[k][s] = !e ? 0.f : REV ? a.W1[(size_t)i * L + l] : a.W2[(size_t)l * M + i] * pf_at(i, N, a.alpha);
        }
    }
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int k = 0; k < NLW; ++k)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int lt = wv * NLW + k, i = 16 * I + c, l = 16 * lt + 4 * g + q;
                const bool e = lt < nlt && i < M && l < L;
                a2[I][4 * k + q] =
                    !e ? 0.f : REV ? a.W2[(size_t)l * M + i] * pf_at(i, N, a.alpha) : a.W1[(size_t)i * L + l];
            }
    const int nchains = a.B * ncs;
    const int id = blockIdx.x * 16 + c;
    const bool exists = id < nchains;
    const int b = exists ? id / ncs : 0, cc = exists ? id % ncs : 0;
    const bool ok = exists && (!active || active[b]);
    const int s0 = cc * C;
    const int len = ok ? max(min(s0 + C, T) - s0, 0) : 0;
    // steps of the block: the longest chain of its 16 (the same value in every wave)
    int maxlen = len;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) maxlen = max(maxlen, __shfl_xor(maxlen, off, 64));
    maxlen = __builtin_amdgcn_readfirstlane(maxlen);
    const float gm = gamma ? gamma[b] : 1.f;
    const float *zin = REV ? nullptr : cur_iter(zbuf, outbuf, zsel, b);
    float *zout = REV ? outbuf : next_iter(zbuf, outbuf, zsel, b);
    float dg[NI][4];
    v4f dl[NI];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * I + 4 * g + r;
            dg[I][r] = i < M ? a.A[i] * pf_at(i, N, a.alpha) : 0.f;
            dl[I][r] = (ok && i < M) ? carry_in[(size_t)id * MP + i] : 0.f;
        }
    const size_t rowb = (size_t)b * T;
    // row of step t of this chain, and whether its Jacobian exists (reverse: J~_{k+1}, k + 1 < T)
    auto krow = [&](int t) { return REV ? s0 + len - 1 - t : s0 + t; };
    // per step: mask words of the wave's tiles; the right-hand side and (forward) the iterate
    // of the element r = w of every tile (wave w adds the diagonal and right-hand side of that
    // element and writes it), one step ahead
    uint32_t mn[NLW];
    float rn[NI], zn[NI];
    auto fetch = [&](int t) {
        const bool run = t < len;
        const int k = krow(t);
        const int mrow = REV ? k + 1 : k;
        const bool hasj = run && mrow < T;
#pragma unroll
        for (int kk = 0; kk < NLW; ++kk) {
            const int lt = wv * NLW + kk;
            mn[kk] = (hasj && lt < nlt) ? masks[(rowb + mrow) * LW + (lt >> 1)] : 0u;
        }
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            const int i = 16 * I + 4 * g + wv;
            const bool e = run && i < M;
            rn[I] = e ? rhs[(rowb + k) * M + i] : 0.f;
            zn[I] = (!REV && e) ? zin[(rowb + k) * M + i] : 0.f;
        }
    };
    fetch(0);
    uint32_t emax = 0u, zmax = 0u;
    for (int t = 0; t < maxlen; ++t) {
        uint32_t mc[NLW];
        float rcur[NI], zcur[NI];
#pragma unroll
        for (int k = 0; k < NLW; ++k) mc[k] = mn[k];
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            rcur[I] = rn[I];
            zcur[I] = zn[I];
        }
        const int kcur = krow(t);
        // the Jacobian term of this step: always forward; reverse unless k + 1 = T
        const bool hasj = !REV || kcur + 1 < T;
        // latent warm-up step of this lane's chain (P_1 in J~_k, forward, or J~_{k+1}, reverse):
        // the observed latents' entries of y enter neither W2 diag(p) y nor the diagonal term
        // (forward), or the output's observed rows vanish (reverse)
        const bool wdrop = a.tw > 0 && (REV ? kcur + 1 : kcur) <= a.tw && t < len;
        if (!REV && a.tw > 0) {
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (wdrop && 16 * I + 4 * g + r < N) dl[I][r] = 0.f;
        }
        fetch(t + 1);
        v4f u[NLW];
#pragma unroll
        for (int k = 0; k < NLW; ++k) {
            v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q4 = 0; q4 < NS; ++q4) s = mfma16x16x4(a1[k][q4], dl[q4 / 4][q4 % 4], s);
            const int sh = 16 * ((wv * NLW + k) & 1) + 4 * g;
#pragma unroll
            for (int r = 0; r < 4; ++r) s[r] = select_bit(mc[k], sh + r, s[r]);
            u[k] = s;
        }
        v4f p2[NI];
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < NLW; ++k)
#pragma unroll
                for (int q = 0; q < 4; ++q) s = mfma16x16x4(a2[I][4 * k + q], u[k][q], s);
            p2[I] = s;
        }
        const int buf = t & 1;
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            v4f ct;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool own = r == wv;
                const bool jon = hasj && !(REV && wdrop && 16 * I + 4 * g + r < N);
                const float jv = jon ? gm * (own ? fmaf(dg[I][r], dl[I][r], p2[I][r]) : p2[I][r]) : 0.f;
                ct[r] = own ? fmaf(rhs_sign, rcur[I], jv) : jv;
            }
            red[buf][wv][I][lane] = ct;
        }
        lds_barrier();
#pragma unroll
        for (int I = 0; I < NI; ++I) {
            v4f s = red[buf][0][I][lane];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                const v4f o = red[buf][w][I][lane];
#pragma unroll
                for (int r = 0; r < 4; ++r) s[r] = s[r] + o[r];
            }
            dl[I] = s;
        }
        if (t < len) {
#pragma unroll
            for (int I = 0; I < NI; ++I) {
                const int i = 16 * I + 4 * g + wv;
                if (i < M) {
                    const v4f d = dl[I];
                    const float y = wv == 0 ? d[0] : wv == 1 ? d[1] : wv == 2 ? d[2] : d[3];
                    if (REV) {
                        zout[(rowb + kcur) * M + i] = y;
                    } else {
                        const float zo = zcur[I];
                        zout[(rowb + kcur) * M + i] = zo + y;
                        const uint32_t ab = abs_bits(y), zb = abs_bits(zo);
                        emax = emax > ab ? emax : ab;
                        zmax = zmax > zb ? zmax : zb;
                    }
                }
            }
        }
    }
    if (REV) return;
    // per-chain maxima: the lane groups, then the 4 waves (through the LDS of the last step,
    // whose reads are done once every wave has passed this barrier)
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
        const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
        emax = emax > o ? emax : o;
        zmax = zmax > oz ? zmax : oz;
    }
    __shared__ uint32_t mx[4][16][2];
    if (g == 0) {
        mx[wv][c][0] = emax;
        mx[wv][c][1] = zmax;
    }
    lds_barrier();
    if (wv != 0) return;
    if (g == 0 && ok) {
#pragma unroll
        for (int w = 1; w < 4; ++w) {
            emax = emax > mx[w][c][0] ? emax : mx[w][c][0];
            zmax = zmax > mx[w][c][1] ? zmax : mx[w][c][1];
        }
        if (!fc.seq) {   // reduced per sequence by the pass-end control
            chain_bits[id] = emax;
            chain_bits[(size_t)nchains + id] = zmax;
        }
    }
    if (!fc.seq) return;
    // fused pass-end control: lane 0 gathers the 16 chains' maxima and arrives once per
    // sequence they belong to (chains of a sequence that is not running do not arrive)
    uint32_t em[16], zm[16];
    bool okc[16];
#pragma unroll
    for (int n = 0; n < 16; ++n) {
        em[n] = (uint32_t)__shfl((int)emax, n, 64);
        zm[n] = (uint32_t)__shfl((int)zmax, n, 64);
        okc[n] = __shfl((int)ok, n, 64) != 0;
    }
    if (lane != 0) return;
    const int chain0 = blockIdx.x * 16;
    for (int n = 0; n < 16; ++n) {
        if (!okc[n]) continue;
        const int bn = (chain0 + n) / ncs;
        if (n > 0 && okc[n - 1] && (chain0 + n - 1) / ncs == bn) continue;   // counted with its first chain
        uint32_t E = 0u, Z = 0u;
        int cnt = 0;
        for (int m2 = n; m2 < 16 && okc[m2] && (chain0 + m2) / ncs == bn; ++m2) {
            E = E > em[m2] ? E : em[m2];
            Z = Z > zm[m2] ? Z : zm[m2];
            ++cnt;
        }
        seq_arrive(fc, bn, cnt, ncs, E, Z);
    }
}

// ---------------------------------------------------------------------------------------
// residual and hidden masks of a Newton pass on the matrix cores.  A wave owns a tile of 16
// rows (b, s), the 16 columns of its products; W2 (row l, column i), W1 (row i, column l) and
// h2 sit in LDS and serve as A operands.  Per 16-unit hidden tile lt:
//   u   = W2[tile lt, :] z~ + h2     B = z~ of the rows (lane (g, c): z~[row c][16j + 4g + q])
//   m   = u > 0 (the 4 lane groups' bits ORed into the row's mask word), v = relu(u)
//   F  += W1[:, tile lt] v           B = v in its accumulator layout
// and F = A z~ + F + h1, r = z - F.  No barrier inside the loop over tiles.  The sums round as
// the matrix cores do, so a decision with u within rounding of 0 may differ from the
// fixed-order float32 one of k_resjac_shplrnn; these masks serve only the Newton passes (the
// masks a caller receives and the adjoint's come from k_resjac_shplrnn).
// ---------------------------------------------------------------------------------------
static int shf_LQ(int L) { return shf_LP(L) + 4; }

size_t shf_resjac_lds(int M, int L) {
    const int MP = padded_dim(M), LP = shf_LP(L);
    return ((size_t)LP * (MP + 4) + (size_t)MP * shf_LQ(L) + LP) * sizeof(float);
}

template <int MP>
__global__ __launch_bounds__(256) void k_resjac_shmfma(const ShArgs a, const float *zbuf, const float *zalt,
                                                       const int *__restrict__ zsel, float *__restrict__ r_out,
                                                       uint32_t *__restrict__ masks, const int *__restrict__ active,
                                                       int LP, uint32_t *mark, uint32_t pass_no) {
    constexpr int NI = MP / 16, MQ = MP + 4;
    extern __shared__ __align__(16) float smem[];
    // the pass's first kernel: block 0 marks its start (every earlier pass is complete)
    if (mark && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(mark, pass_no, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const int M = a.M, L = a.L, T = a.T, N = a.N, LQ = LP + 4;
    float *w2s = smem;             // [LP][MQ]
    float *w1s = w2s + LP * MQ;    // [MP][LQ]
    float *h2s = w1s + MP * LQ;    // [LP]
    const int tid = threadIdx.x;
    for (int e = tid; e < LP * MQ; e += 256) {
        const int l = e / MQ, i = e % MQ;
        w2s[e] = (l < L && i < M) ? a.W2[(size_t)l * M + i] : 0.f;
    }
    for (int e = tid; e < MP * LQ; e += 256) {
        const int i = e / LQ, l = e % LQ;
        w1s[e] = (i < M && l < L) ? a.W1[(size_t)i * L + l] : 0.f;
    }
    for (int e = tid; e < LP; e += 256) h2s[e] = (e < L && a.h2) ? a.h2[e] : 0.f;
    __syncthreads();
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32, nlt = LP / 16;
    const float p = __fsub_rn(1.0f, a.alpha);
    float dA[NI][4], h1v[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * I + 4 * g + r;
            dA[I][r] = i < M ? a.A[i] : 0.f;
            h1v[I][r] = (i < M && a.h1) ? a.h1[i] : 0.f;
        }
    const long total = (long)a.B * T;
    const long ntiles = (total + 15) / 16;
    const long nw = (long)gridDim.x * 4;
    // The inputs of a tile for row c, latents i = 16j + 4g + q: z_{s-1} (or the initial state at
    // s = 0) and x_s, combined into z~ as k_resjac_shplrnn does, and z_s.  Every lane loads from a
    // valid address (rows past the end, inactive sequences and latents past M read row 0 /
    // latent 0 and are zeroed after), so the loads carry no branches and the next tile's, issued
    // at the top of a tile, are waited for only when the tile ends.
    struct RowIn {   // (sequence, step) of row c of a tile and the sequence's control words
        int b, s, sel, act;
        bool inr;
    };
    struct TileIn {
        float zp[NI][4], xs[NI][4], zc[NI][4];
        int s;
        bool ok;
    };
    // stage 1, two tiles ahead: the row's position and its control words (loads in flight)
    auto rowin = [&](long tile, RowIn &ri) {
        const long rowc = tile * 16 + c;
        ri.b = 0;
        ri.s = 0;
        ri.inr = tile < ntiles && rowc < total;
        if (ri.inr) row_at(row_base(tile * 16, T), c, T, ri.b, ri.s);
        ri.sel = zsel ? zsel[ri.b] : 0;
        ri.act = active ? active[ri.b] : 1;
    };
    // stage 2, one tile ahead: the inputs, at addresses from the control words loaded a tile ago
    auto fetch = [&](const RowIn &ri, TileIn &in) {
        const int b = ri.b, s = ri.s;
        in.ok = ri.inr && ri.act != 0;
        in.s = s;
        const float *z = ri.sel ? zalt : zbuf;
        const size_t rp = (size_t)b * T + (s > 0 ? s - 1 : 0), rc = (size_t)b * T + s;
        const size_t xr = ((size_t)b * (T + 1) + s) * (size_t)(N > 0 ? N : 1);
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = 16 * j + 4 * g + q, ic = i < M ? i : 0;
                const float zpv = z[rp * M + ic];
                const float z0v = a.z0 ? a.z0[(size_t)b * M + ic] : 0.f;
                in.zp[j][q] = s > 0 ? zpv : z0v;
                in.xs[j][q] = N > 0 ? a.x[xr + (i < N ? i : 0)] : 0.f;
                in.zc[j][q] = z[rc * M + ic];
            }
    };
    const long t0w = (long)blockIdx.x * 4 + wv;
    RowIn r1, r2;
    TileIn cur, nxt;
    rowin(t0w, r1);
    fetch(r1, cur);
    rowin(t0w + nw, r1);
    for (long tile = t0w; tile < ntiles; tile += nw) {
        rowin(tile + 2 * nw, r2);
        fetch(r1, nxt);
        const long rowc = tile * 16 + c;
        const bool rok = cur.ok;
        const int s = cur.s;
        float zt[NI][4], zc[NI][4];
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = 16 * j + 4 * g + q;
                float v;
                if (s == 0)   // the initial state: z0, or [x_0; 0]
                    v = a.z0 ? cur.zp[j][q] : (i < N ? cur.xs[j][q] : 0.f);
                else if (i < N && s <= a.tw)   // latent warm-up: alpha_s = 1
                    v = cur.xs[j][q];
                else
                    v = i < N ? __fadd_rn(__fmul_rn(p, cur.zp[j][q]), __fmul_rn(a.alpha, cur.xs[j][q])) : cur.zp[j][q];
                const bool e = rok && i < M;
                zt[j][q] = e ? v : 0.f;
                zc[j][q] = e ? cur.zc[j][q] : 0.f;
            }
        // a tile whose sequences have all stopped (a pass queued past their convergence) does no
        // work (the branch is wave-uniform)
        if (__builtin_amdgcn_ballot_w64(rok) != 0ull) {
            v4f F[NI];
    #pragma unroll
            for (int I = 0; I < NI; ++I) F[I] = (v4f){0.f, 0.f, 0.f, 0.f};
            for (int w = 0; w < LW; ++w) {
                uint32_t word = 0u;
    #pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int lt = 2 * w + h;
                    if (lt >= nlt) break;
                    const float4 hq = *reinterpret_cast<const float4 *>(h2s + 16 * lt + 4 * g);
                    v4f u = {hq.x, hq.y, hq.z, hq.w};
    #pragma unroll
                    for (int j = 0; j < NI; ++j) {
                        const float4 aq = *reinterpret_cast<const float4 *>(w2s + (16 * lt + c) * MQ + 16 * j + 4 * g);
                        u = mfma16x16x4(aq.x, zt[j][0], u);
                        u = mfma16x16x4(aq.y, zt[j][1], u);
                        u = mfma16x16x4(aq.z, zt[j][2], u);
                        u = mfma16x16x4(aq.w, zt[j][3], u);
                    }
    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const bool on = u[r] > 0.f;
                        word |= (on ? 1u : 0u) << (16 * h + 4 * g + r);
                        u[r] = on ? u[r] : 0.f;
                    }
    #pragma unroll
                    for (int I = 0; I < NI; ++I) {
                        const float4 aq = *reinterpret_cast<const float4 *>(w1s + (16 * I + c) * LQ + 16 * lt + 4 * g);
                        F[I] = mfma16x16x4(aq.x, u[0], F[I]);
                        F[I] = mfma16x16x4(aq.y, u[1], F[I]);
                        F[I] = mfma16x16x4(aq.z, u[2], F[I]);
                        F[I] = mfma16x16x4(aq.w, u[3], F[I]);
                    }
                }
                word |= (uint32_t)__shfl_xor((int)word, 16, 64);
                word |= (uint32_t)__shfl_xor((int)word, 32, 64);
                if (g == 0 && rok) masks[(size_t)rowc * LW + w] = word;
            }
            if (rok) {
    #pragma unroll
                for (int I = 0; I < NI; ++I)
    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = 16 * I + 4 * g + r;
                        if (i < M) r_out[(size_t)rowc * M + i] = zc[I][r] - (fmaf(dA[I][r], zt[I][r], F[I][r]) + h1v[I][r]);
                    }
            }
        }
        cur = nxt;
        r1 = r2;
    }
}

int launch_resjac_shmfma(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *r,
                         uint32_t *masks, const int *active, hipStream_t st, uint32_t *mark, uint32_t pass_no) {
    const int MP = padded_dim(a.M);
    if (!shfused_supported(a.M, a.L) || a.zt) return DEER_ERR_INVALID_ARG;
    const size_t lds = shf_resjac_lds(a.M, a.L);
    if (lds > 80 * 1024) return DEER_ERR_INVALID_ARG;
    const long ntiles = ((long)a.B * a.T + 15) / 16;
    // two resident blocks per CU (LDS), each wave walking its share of the tiles
    const long want = (ntiles + 3) / 4;
    const int grid = (int)(want < 512 ? want : 512);
    const int LP = shf_LP(a.L);
    KTimer kt("k_resjac_shmfma", st);
#define RJM(MPV) \
    hipLaunchKernelGGL((k_resjac_shmfma<MPV>), dim3(grid), dim3(256), lds, st, a, z, zalt, zsel, r, masks, active, LP, \
                       mark, pass_no)
    if (MP == 16) RJM(16); else if (MP == 32) RJM(32); else RJM(64);
#undef RJM
    DEER_LAUNCH_CHECK("k_resjac_shmfma");
    return DEER_OK;
}

int launch_chunk_product_shfused(bool rev, const ShArgs &a, const uint32_t *masks, const float *rhs,
                                 float rhs_sign, const float *gamma, float *P, float *v, const int *active, int C,
                                 int ncs, hipStream_t st) {
    const int MP = padded_dim(a.M);
    if (!shfused_supported(a.M, a.L) || (rev && (gamma || active))) return DEER_ERR_INVALID_ARG;
    const int nch = a.B * ncs;
    const int grid = (nch + 3) / 4;
    const int LP = shf_LP(a.L);
    const size_t lds = shfused_product_lds(a.M, a.L);
    KTimer kt(rev ? "k_chunk_product_shfused_rev" : "k_chunk_product_shfused", st);
#define CPS(MPV, NTV)                                                                                             \
    hipLaunchKernelGGL((k_chunk_product_shfused<MPV, NTV>), dim3(grid), dim3(256), lds, st, a, masks, rhs, rhs_sign, \
                       gamma, P, v, active, C, ncs, LP)
#define CPR(MPV, NTV)                                                                                            \
    hipLaunchKernelGGL((k_chunk_product_shfused_rev<MPV, NTV>), dim3(grid), dim3(256), lds, st, a, masks, rhs, \
                       rhs_sign, P, v, C, ncs, LP)
    if (rev) {
        if (MP == 16) CPR(16, 4); else if (MP == 32) CPR(32, 4); else CPR(64, 1);
    } else {
        if (MP == 16) CPS(16, 4); else if (MP == 32) CPS(32, 4); else CPS(64, 1);
    }
#undef CPR
#undef CPS
    DEER_LAUNCH_CHECK("k_chunk_product_shfused");
    return DEER_OK;
}

int launch_fixup_shjvp(bool rev, const ShArgs &a, const uint32_t *masks, const float *rhs, float rhs_sign,
                       const float *gamma, const float *carry_in, float *z, float *out, const int *zsel,
                       uint32_t *chain_bits, const int *active, int C, int ncs, hipStream_t st, const FusedCtl *fc) {
    const int MP = padded_dim(a.M);
    if (!shfused_supported(a.M, a.L) || (fc && (rev || !active))) return DEER_ERR_INVALID_ARG;
    const FusedCtl fcv = fc ? *fc : FusedCtl{};
    const int nch = a.B * ncs;
    const int grid = (nch + 15) / 16;
    const int nlw = shf_nlw(a.L);
    KTimer kt(rev ? "k_fixup_shjvp_rev" : "k_fixup_shjvp", st);
#define FXJ(MPV, NL, RV)                                                                                         \
    hipLaunchKernelGGL((k_fixup_shjvp<MPV, NL, RV>), dim3(grid), dim3(256), 0, st, a, masks, rhs, rhs_sign, gamma, \
                       carry_in, z, out, zsel, chain_bits, active, C, ncs, fcv)
    // shfused_supported bounds NLW * MP / 2 (the A fragments per lane) by 64
#define FXJ_ALL(RV)                                                                                                  \
    if (MP == 16) {                                                                                                  \
        if (nlw == 1) FXJ(16, 1, RV); else if (nlw == 2) FXJ(16, 2, RV); else if (nlw == 4) FXJ(16, 4, RV);          \
        else FXJ(16, 8, RV);                                                                                         \
    } else if (MP == 32) {                                                                                           \
        if (nlw == 1) FXJ(32, 1, RV); else if (nlw == 2) FXJ(32, 2, RV); else FXJ(32, 4, RV);                        \
    } else {                                                                                                         \
        if (nlw == 1) FXJ(64, 1, RV); else FXJ(64, 2, RV);                                                           \
    }
    if (rev) { FXJ_ALL(true) } else { FXJ_ALL(false) }
#undef FXJ_ALL
#undef FXJ
    DEER_LAUNCH_CHECK("k_fixup_shjvp");
    return DEER_OK;
}

}  // namespace deer
