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

bool shfused_supported(int M, int L) {
    const int MP = padded_dim(M);
    if (MP > 64 || L <= 0) return false;
    if (shfused_product_lds(M, L) > 80 * 1024) return false;   // two blocks per CU
    const int nlw = shf_nlw(L);
    // fix-up A fragments in registers: NLW * (MP / 4) + (MP / 16) * 4 NLW floats per lane
    return nlw > 0 && nlw * (MP / 4 + MP / 4) <= 64;
}

// ---------------------------------------------------------------------------------------
// chunk product.  LDS: w2t [MP][LQ] = (W2 diag(p))^T (row i, column l) and w1s [MP][LQ] = W1
// (row j, column l), LQ = LP + 4 (rows of a 16-lane group fall on different banks).
// jt tile (I, Jt) of step nt: lane (g, c) element r = J~^T[16I + 4g + r][16Jt + c]
//   = J~[16Jt + c][16I + 4g + r], which is the A fragment of row tile Jt, k-step 4I + r of
// the product kernel (lane (g, c) holds J~[16I' + c][16j + 4g + q]).
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
    const int tid = threadIdx.x;
    for (int e = tid; e < MP * LQ; e += 256) {
        const int i = e / LQ, l = e % LQ;
        const bool ok = i < M && l < L;
        w2t[e] = ok ? a.W2[(size_t)l * M + i] * pf_at(i, N, a.alpha) : 0.f;
        w1s[e] = ok ? a.W1[(size_t)i * L + l] : 0.f;
    }
    __syncthreads();
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
    float dg[NI];   // A_i p_i of row i = 16 I + c (the diagonal of the A fragments of row tile I)
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
        // right-hand sides of the NT steps (lanes of column 0), loaded before the formation
        float rc[NT][NI][4];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = 16 * I + 4 * g + r;
                    rc[nt][I][r] = (t0 + nt < len && c == 0 && row < M) ? rhs[(row0 + t0 + nt) * M + row] : 0.f;
                }
        v4f jt[NT][NI][NI];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt) jt[nt][I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
        // mask words: one per pair of 16-unit k tiles, loaded a pair ahead
        uint32_t mw[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mw[nt] = t0 + nt < len ? masks[(row0 + t0 + nt) * LW] : 0u;
        for (int jp = 0; jp < njl; jp += 2) {
            uint32_t mc[NT];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                mc[nt] = mw[nt];
                const int wn = (jp >> 1) + 1;
                mw[nt] = (t0 + nt < len && wn < LW) ? masks[(row0 + t0 + nt) * LW + wn] : 0u;
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int j = jp + h;
                if (j >= njl) break;
                float4 av[NI], bv[NI];
#pragma unroll
                for (int I = 0; I < NI; ++I)
                    av[I] = *reinterpret_cast<const float4 *>(w2t + (16 * I + c) * LQ + 16 * j + 4 * g);
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt)
                    bv[Jt] = *reinterpret_cast<const float4 *>(w1s + (16 * Jt + c) * LQ + 16 * j + 4 * g);
                const int sh = 16 * h + 4 * g;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    if (t0 + nt >= len) continue;
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
            }
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (t0 + nt >= len) break;
            // A fragments: row tile I, k-step s = 4j + q holds J~[16I + c][16j + 4g + q]
            float ac[NI][NS];
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        float v = jt[nt][j][I][q];
                        if (I == j && c == 4 * g + q) v = v + dg[I];
                        ac[I][4 * j + q] = gm * v;
                    }
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
// fix-up (forward Newton update: next iterate = current + Delta, per-chain max |Delta| and
// max |z|).  Block = 16 chains (column c = lane & 15) x 4 waves; wave w owns the l tiles
// lt = NLW w + k.  Per step, with Delta tiles dl[I] (lane (g, c) element r = Delta[16I + 4g + r]
// of chain c, replicated in all 4 waves):
//   u[k]  = (W2 diag(p))[tile lt, :] Delta        A = W2 p rows, B = dl (k-permuted layout)
//   u[k] *= m_t                                    the mask bits of l = 16 lt + 4g + r
//   p2[I] = W1[tile I, tiles of the wave] u        A = W1 rows, B = u (the same layout)
// The waves' contributions gamma p2 (wave 0: gamma (p2 + A p Delta) + s r_t) are summed in LDS
// in a fixed order, so every wave holds the same next Delta.
// ---------------------------------------------------------------------------------------
template <int MP, int NLW>
__global__ __launch_bounds__(256) void k_fixup_shjvp(const ShArgs a, const uint32_t *__restrict__ masks,
                                                     const float *__restrict__ rhs, float rhs_sign,
                                                     const float *__restrict__ gamma,
                                                     const float *__restrict__ carry_in, float *zbuf, float *outbuf,
                                                     const int *__restrict__ zsel, uint32_t *__restrict__ chain_bits,
                                                     const int *__restrict__ active, int C, int ncs) {
    constexpr int NI = MP / 16, NS = MP / 4;
    __shared__ v4f red[2][4][NI][64];
    const int tid = threadIdx.x, wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4,
              c = lane & 15;
    const int M = a.M, L = a.L, T = a.T, N = a.N;
    const int LW = (L + 31) / 32, nlt = (L + 15) / 16;
    float a1[NLW][NS], a2[NI][4 * NLW];
#pragma unroll
    for (int k = 0; k < NLW; ++k) {
        const int lt = wv * NLW + k, l = 16 * lt + c;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int i = 16 * (s / 4) + 4 * g + (s % 4);
            a1[k][s] = (lt < nlt && l < L && i < M) ? a.W2[(size_t)l * M + i] * pf_at(i, N, a.alpha) : 0.f;
        }
    }
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int k = 0; k < NLW; ++k)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int lt = wv * NLW + k, i = 16 * I + c, l = 16 * lt + 4 * g + q;
                a2[I][4 * k + q] = (lt < nlt && i < M && l < L) ? a.W1[(size_t)i * L + l] : 0.f;
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
    const float *zin = cur_iter(zbuf, outbuf, zsel, b);
    float *zout = next_iter(zbuf, outbuf, zsel, b);
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
    const size_t rowb = (size_t)b * T + s0;
    // per step: mask words of the wave's tiles (all waves); r_t and z_t (wave 0), one step ahead
    uint32_t mn[NLW];
    float rn[NI][4], zn[NI][4];
    auto fetch = [&](int t) {
        const bool run = t < len;
#pragma unroll
        for (int k = 0; k < NLW; ++k) {
            const int lt = wv * NLW + k;
            mn[k] = (run && lt < nlt) ? masks[(rowb + t) * LW + (lt >> 1)] : 0u;
        }
        if (wv == 0) {
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 16 * I + 4 * g + r;
                    const bool e = run && i < M;
                    rn[I][r] = e ? rhs[(rowb + t) * M + i] : 0.f;
                    zn[I][r] = e ? zin[(rowb + t) * M + i] : 0.f;
                }
        }
    };
    fetch(0);
    uint32_t emax = 0u, zmax = 0u;
    for (int t = 0; t < maxlen; ++t) {
        uint32_t mc[NLW];
        float rcur[NI][4], zcur[NI][4];
#pragma unroll
        for (int k = 0; k < NLW; ++k) mc[k] = mn[k];
#pragma unroll
        for (int I = 0; I < NI; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                rcur[I][r] = rn[I][r];
                zcur[I][r] = zn[I][r];
            }
        fetch(t + 1);
        // u = (W2 diag(p)) Delta on this wave's hidden tiles, masked
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
        // W1 on the masked hidden values of this wave
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
                if (wv == 0)
                    ct[r] = fmaf(rhs_sign, rcur[I][r], gm * fmaf(dg[I][r], dl[I][r], p2[I][r]));
                else
                    ct[r] = gm * p2[I][r];
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
        if (wv == 0 && t < len) {
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 16 * I + 4 * g + r;
                    if (i < M) {
                        const float y = dl[I][r], zo = zcur[I][r];
                        zout[(rowb + t) * M + i] = zo + y;
                        const uint32_t ab = abs_bits(y), zb = abs_bits(zo);
                        emax = emax > ab ? emax : ab;
                        zmax = zmax > zb ? zmax : zb;
                    }
                }
        }
    }
    if (wv != 0) return;
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)emax, off, 64);
        const uint32_t oz = (uint32_t)__shfl_xor((int)zmax, off, 64);
        emax = emax > o ? emax : o;
        zmax = zmax > oz ? zmax : oz;
    }
    if (ok && g == 0) {   // per-chain maxima, reduced per sequence by the pass-end control
        chain_bits[id] = emax;
        chain_bits[(size_t)nchains + id] = zmax;
    }
}

int launch_chunk_product_shfused(const ShArgs &a, const uint32_t *masks, const float *rhs, float rhs_sign,
                                 const float *gamma, float *P, float *v, const int *active, int C, int ncs,
                                 hipStream_t st) {
    const int MP = padded_dim(a.M);
    if (!shfused_supported(a.M, a.L)) return DEER_ERR_INVALID_ARG;
    const int nch = a.B * ncs;
    const int grid = (nch + 3) / 4;
    const int LP = shf_LP(a.L);
    const size_t lds = shfused_product_lds(a.M, a.L);
    KTimer kt("k_chunk_product_shfused", st);
#define CPS(MPV, NTV)                                                                                             \
    hipLaunchKernelGGL((k_chunk_product_shfused<MPV, NTV>), dim3(grid), dim3(256), lds, st, a, masks, rhs, rhs_sign, \
                       gamma, P, v, active, C, ncs, LP)
    if (MP == 16) CPS(16, 4); else if (MP == 32) CPS(32, 4); else CPS(64, 1);
#undef CPS
    DEER_LAUNCH_CHECK("k_chunk_product_shfused");
    return DEER_OK;
}

int launch_fixup_shjvp(const ShArgs &a, const uint32_t *masks, const float *rhs, float rhs_sign, const float *gamma,
                       const float *carry_in, float *z, float *out, const int *zsel, uint32_t *chain_bits,
                       const int *active, int C, int ncs, hipStream_t st) {
    const int MP = padded_dim(a.M);
    if (!shfused_supported(a.M, a.L)) return DEER_ERR_INVALID_ARG;
    const int nch = a.B * ncs;
    const int grid = (nch + 15) / 16;
    const int nlw = shf_nlw(a.L);
    KTimer kt("k_fixup_shjvp", st);
#define FXJ(MPV, NL) \
    hipLaunchKernelGGL((k_fixup_shjvp<MPV, NL>), dim3(grid), dim3(256), 0, st, a, masks, rhs, rhs_sign, gamma, carry_in, \
                       z, out, zsel, chain_bits, active, C, ncs)
    // shfused_supported bounds NLW * MP / 2 (the A fragments per lane) by 64
    if (MP == 16) {
        if (nlw == 1) FXJ(16, 1); else if (nlw == 2) FXJ(16, 2); else if (nlw == 4) FXJ(16, 4); else FXJ(16, 8);
    } else if (MP == 32) {
        if (nlw == 1) FXJ(32, 1); else if (nlw == 2) FXJ(32, 2); else FXJ(32, 4);
    } else {
        if (nlw == 1) FXJ(64, 1); else FXJ(64, 2);
    }
#undef FXJ
    DEER_LAUNCH_CHECK("k_fixup_shjvp");
    return DEER_OK;
}

}  // namespace deer
