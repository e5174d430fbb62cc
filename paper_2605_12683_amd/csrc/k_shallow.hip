// Shallow PLRNN path of GTF-DEER on gfx950 (eq. shplrnn_nonlinear with V = W2, b = h2):
//   u_t  = W2 z~_{t-1} + h2                     (L hidden units)
//   z_t  = diag(A) z~_{t-1} + W1 relu(u_t) + h1
//   J~_t = (diag(A) + W1 diag(m_t) W2) P_alpha,  m_t = (u_t > 0)
//
//   k_resjac_shplrnn   r_t, F_t and the hidden masks m_t.  u is accumulated left to right in
//                      float32 from h2 with separate roundings (no fused multiply-add), which
//                      makes the ReLU decision reproducible bit for bit.
//   k_jacform_shplrnn  J~_t for every step on the matrix cores (fp32 MFMA, K = L), written to
//                      HBM for the stored-Jacobian scan.
//   k_grads_shplrnn    per-block partial sums of dA, dW1, dW2, dh1, dh2 from lam (gradients
//                      appendix), reduced in float64 by k_reduce_rows.
#include "common.h"
#include "launch.h"

namespace deer {

__device__ __forceinline__ float p_at(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

// ---------------------------------------------------------------------------------------
// residual + masks.  Block of 256 threads (4 waves), TT rows (b, t) per tile, grid-stride
// over tiles.  The hidden pre-activations u = W2 z~ + h2 that decide the masks are summed on
// the VALU in a fixed order (left to right from h2, a rounding after every multiply and add);
// F = A z~ + W1 relu(u) + h1 is a [M x L] x [L x TT] product on the matrix cores with the
// k range split over the 4 waves and the partial tiles summed through LDS.
// dynamic LDS: zt[TT][MP] | ru[TT][LQ] | W1[MP][LQ] | partial F tiles [4][NI][64][4]
// (LQ = L rounded up to 16, + 4 so that rows stay 16-byte aligned and spread over banks)
// ---------------------------------------------------------------------------------------
constexpr int SH_TT = 16;

static __host__ __device__ inline int sh_LQ(int L) { return (L + 15) / 16 * 16 + 4; }

template <int MP>
__global__ __launch_bounds__(256) void k_resjac_shplrnn(const ShArgs a, const float *zbuf, const float *zalt,
                                                        const int *__restrict__ zsel, float *__restrict__ F_out,
                                                        float *__restrict__ r_out, uint32_t *__restrict__ masks,
                                                        const int *__restrict__ active) {
    constexpr int NI = MP / 16;
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, LQ = sh_LQ(L);
    float *zt = smem;                    // [SH_TT][MP], zero padded
    float *ru = zt + SH_TT * MP;         // [SH_TT][LQ], zero padded
    float *w1s = ru + SH_TT * LQ;        // [MP][LQ] = W1, zero padded
    v4f *red = reinterpret_cast<v4f *>(w1s + MP * LQ);   // [4][NI][64]
    const int tid = threadIdx.x;
    const int lane = tid & 63, wv = tid >> 6, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    for (int e = tid; e < MP * LQ; e += 256) {
        const int i = e / LQ, l = e % LQ;
        w1s[e] = (i < M && l < L) ? a.W1[i * L + l] : 0.f;
    }
    for (int e = tid; e < SH_TT * LQ; e += 256) ru[e] = 0.f;
    const long total = (long)a.B * T;
    const long ntiles = (total + SH_TT - 1) / SH_TT;
    const int njg = (L + 15) / 16;
    for (long tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const long row0 = tile * SH_TT;
        __syncthreads();
        for (int e = tid; e < SH_TT * MP; e += 256) {
            const int tt = e / MP, i = e % MP;
            const long row = row0 + tt;
            float v = 0.f;
            if (row < total && i < M) {
                const int b = (int)(row / T), s = (int)(row % T);
                v = forced_state(a.x, a.z0, cur_iter(zbuf, zalt, zsel, b), b, s, i, T, M, a.N, a.alpha);
            }
            zt[e] = v;
        }
        __syncthreads();
        // hidden pre-activations: left to right in k from h2, separate roundings.  The zero
        // padding adds exact zeros, so the value is the one of the unpadded sum.
        for (int jb = 0; jb < L; jb += 256) {
            const int j = jb + tid;
            const bool jok = j < L;
            float w2r[MP];
#pragma unroll
            for (int k = 0; k < MP; ++k) w2r[k] = (jok && k < M) ? a.W2[(size_t)j * M + k] : 0.f;
            const float h2j = (jok && a.h2) ? a.h2[j] : 0.f;
            // RG rows at a time: independent chains interleaved (each sum is serial in k)
            constexpr int RG = 4;
            for (int tt0 = 0; tt0 < SH_TT; tt0 += RG) {
                float u[RG];
#pragma unroll
                for (int q = 0; q < RG; ++q) u[q] = h2j;
#pragma unroll
                for (int k = 0; k < MP; ++k)
#pragma unroll
                    for (int q = 0; q < RG; ++q) u[q] = __fadd_rn(u[q], __fmul_rn(w2r[k], zt[(tt0 + q) * MP + k]));
#pragma unroll
                for (int q = 0; q < RG; ++q) {
                    const int tt = tt0 + q;
                    const bool pos = jok && u[q] > 0.f;
                    if (jok) ru[tt * LQ + j] = pos ? u[q] : 0.f;
                    const uint64_t bal = __ballot(pos);
                    const long row = row0 + tt;
                    if (masks && row < total && (lane == 0 || lane == 32)) {
                        const int b = (int)(row / T);
                        if (!active || active[b]) {
                            const int word = (jb + tid) / 32;
                            if (word < LW) masks[(size_t)row * LW + word] = (uint32_t)(bal >> lane);
                        }
                    }
                }
            }
        }
        __syncthreads();
        // F^T tile [MP x 16 rows] = W1 relu(U)^T, this wave's share of the k range; lane (g, c)
        // ends with F^T[16I + 4g + r][row c]; k-step (jg, q) uses k = 16 jg + 4g + q in group g
        v4f fa[NI];
#pragma unroll
        for (int I = 0; I < NI; ++I) fa[I] = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int jg = wv; jg < njg; jg += 4) {
            const float4 bq = *reinterpret_cast<const float4 *>(ru + c * LQ + 16 * jg + 4 * g);
#pragma unroll
            for (int I = 0; I < NI; ++I) {
                const float4 aq = *reinterpret_cast<const float4 *>(w1s + (16 * I + c) * LQ + 16 * jg + 4 * g);
                fa[I] = mfma16x16x4(aq.x, bq.x, fa[I]);
                fa[I] = mfma16x16x4(aq.y, bq.y, fa[I]);
                fa[I] = mfma16x16x4(aq.z, bq.z, fa[I]);
                fa[I] = mfma16x16x4(aq.w, bq.w, fa[I]);
            }
        }
#pragma unroll
        for (int I = 0; I < NI; ++I) red[(wv * NI + I) * 64 + lane] = fa[I];
        __syncthreads();
        if (wv == 0) {
            const long row = row0 + c;
            const bool rok = row < total && (!active || active[row / T]);
            if (rok) {
                const float *zc = cur_iter(zbuf, zalt, zsel, (int)(row / T));
#pragma unroll
                for (int I = 0; I < NI; ++I) {
                    v4f sum = red[I * 64 + lane];
#pragma unroll
                    for (int w = 1; w < 4; ++w) {
                        const v4f o = red[(w * NI + I) * 64 + lane];
                        sum[0] += o[0]; sum[1] += o[1]; sum[2] += o[2]; sum[3] += o[3];
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = 16 * I + 4 * g + r;
                        if (i < M) {
                            const float F = fmaf(a.A[i], zt[c * MP + i], sum[r]) + (a.h1 ? a.h1[i] : 0.f);
                            const size_t e2 = (size_t)row * M + i;
                            if (F_out) F_out[e2] = F;
                            if (r_out) r_out[e2] = zc[e2] - F;
                        }
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// forced Jacobians on the matrix cores.  4 waves per block, each wave NT rows at a time.
// LDS: W1 [MP][LP] and (W2 diag(p))^T [MP][LP], zero padded.
// acc tile (I, Jt) of row nt: lane (g, c) element r = J[16I + 4g + r][16Jt + c]
// k-step s = 4j + q pairs k = 16j + 4g + q (lane group g), as in the other MFMA kernels.
// ---------------------------------------------------------------------------------------
template <int MP, int NT>
__global__ __launch_bounds__(256) void k_jacform_shplrnn(const ShArgs a, const uint32_t *__restrict__ masks,
                                                         float *__restrict__ Jout, const int *__restrict__ active,
                                                         const float *__restrict__ gamma, int LP) {
    extern __shared__ __align__(16) float smem[];
    constexpr int NI = MP / 16;
    const int M = a.M, L = a.L, T = a.T, N = a.N;
    const float alpha = a.alpha;
    float *w1s = smem;             // [MP][LP]
    float *w2s = smem + MP * LP;   // [MP][LP] = (W2 diag(p))^T
    const int tid = threadIdx.x;
    for (int e = tid; e < MP * LP; e += 256) {
        const int i = e / LP, l = e % LP;
        const bool ok = i < M && l < L;
        w1s[e] = ok ? a.W1[(size_t)i * L + l] : 0.f;
        w2s[e] = ok ? a.W2[(size_t)l * M + i] * p_at(i, N, alpha) : 0.f;
    }
    __syncthreads();
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    const long total = (long)a.B * T;
    const long ngroups = (total + NT - 1) / NT;
    float dI[NI][4];
#pragma unroll
    for (int I = 0; I < NI; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * I + 4 * g + r;
            dI[I][r] = row < M ? a.A[row] * p_at(row, N, alpha) : 0.f;
        }
    for (long grp = (long)blockIdx.x * 4 + wv; grp < ngroups; grp += (long)gridDim.x * 4) {
        const long row0 = grp * NT;
        bool rok[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const long row = row0 + nt;
            rok[nt] = row < total && (!active || active[row / T]);
        }
        v4f acc[NT][NI][NI];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt) acc[nt][I][Jt] = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int j = 0; j < LP / 16; ++j) {
            float4 av[NI], bv[NI];
#pragma unroll
            for (int I = 0; I < NI; ++I) av[I] = *reinterpret_cast<const float4 *>(w1s + (16 * I + c) * LP + 16 * j + 4 * g);
#pragma unroll
            for (int Jt = 0; Jt < NI; ++Jt) bv[Jt] = *reinterpret_cast<const float4 *>(w2s + (16 * Jt + c) * LP + 16 * j + 4 * g);
            const int word = (16 * j) >> 5, sh = 16 * (j & 1) + 4 * g;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                if (!rok[nt]) continue;
                const uint32_t w = masks[(size_t)(row0 + nt) * LW + word];
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt) {
                    const float b0 = select_bit(w, sh + 0, bv[Jt].x), b1 = select_bit(w, sh + 1, bv[Jt].y);
                    const float b2 = select_bit(w, sh + 2, bv[Jt].z), b3 = select_bit(w, sh + 3, bv[Jt].w);
#pragma unroll
                    for (int I = 0; I < NI; ++I) {
                        v4f t = acc[nt][I][Jt];
                        t = mfma16x16x4(av[I].x, b0, t);
                        t = mfma16x16x4(av[I].y, b1, t);
                        t = mfma16x16x4(av[I].z, b2, t);
                        t = mfma16x16x4(av[I].w, b3, t);
                        acc[nt][I][Jt] = t;
                    }
                }
            }
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (!rok[nt]) continue;
            float *Jp = Jout + (size_t)(row0 + nt) * M * M;
            // damping of the linearisation of this sequence (1 = exact Newton)
            const float gm = gamma ? gamma[(row0 + nt) / T] : 1.f;
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = 16 * I + 4 * g + r, col = 16 * Jt + c;
                        if (row < M && col < M)
                            Jp[row * M + col] = gm * (acc[nt][I][Jt][r] + (row == col ? dI[I][r] : 0.f));
                    }
        }
    }
}

// ---------------------------------------------------------------------------------------
// parameter gradients.  blockDim = roundup(L, 64) threads, thread l owns hidden unit l:
//   dW1[:, l] += lam_t relu(u_t)_l,   dW2[l, :] += delta_t,l z~_t,   dh2_l += delta_t,l
//   delta_t = (W1^T lam_t) * m_t ;  threads i < M also own dA_i, dh1_i.
// Partials per block: [M*L (dW1, row-major) | L*M (dW2) | L (dh2) | M (dA) | M (dh1)].
// ---------------------------------------------------------------------------------------
constexpr int SHG_TT = 32;
constexpr int SHG_THREADS = 256;

template <int MP>
__global__ __launch_bounds__(SHG_THREADS) void k_grads_shplrnn(const ShArgs a, const float *__restrict__ z,
                                                               const float *__restrict__ lam,
                                                               const uint32_t *__restrict__ masks,
                                                               float *__restrict__ part) {
    __shared__ __align__(16) float zt[SHG_TT][MP];
    __shared__ __align__(16) float lm[SHG_TT][MP];
    const int M = a.M, L = a.L, T = a.T;
    const int tid = threadIdx.x;
    const int l = blockIdx.y * SHG_THREADS + tid;     // hidden unit owned by this thread
    const bool lok = l < L;
    const bool own_latent = blockIdx.y == 0 && tid < M;
    const int LW = (L + 31) / 32;
    float w2r[MP], w1c[MP], dW1c[MP], dW2r[MP];
#pragma unroll
    for (int k = 0; k < MP; ++k) {
        w2r[k] = (lok && k < M) ? a.W2[(size_t)l * M + k] : 0.f;
        w1c[k] = (lok && k < M) ? a.W1[(size_t)k * L + l] : 0.f;
        dW1c[k] = 0.f;
        dW2r[k] = 0.f;
    }
    const float h2l = (lok && a.h2) ? a.h2[l] : 0.f;
    float dh2 = 0.f, dA = 0.f, dh1 = 0.f;
    const long total = (long)a.B * T;
    const long ntiles = (total + SHG_TT - 1) / SHG_TT;
    for (long tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const long row0 = tile * SHG_TT;
        __syncthreads();
        for (int e = tid; e < SHG_TT * MP; e += SHG_THREADS) {
            const int tt = e / MP, i = e % MP;
            const long row = row0 + tt;
            float vz = 0.f, vl = 0.f;
            if (row < total && i < M) {
                const int b = (int)(row / T), s = (int)(row % T);
                vz = forced_state(a.x, a.z0, z, b, s, i, T, M, a.N, a.alpha);
                vl = lam[(size_t)row * M + i];
            }
            zt[tt][i] = vz;
            lm[tt][i] = vl;
        }
        __syncthreads();
        if (own_latent) {
            for (int tt = 0; tt < SHG_TT; ++tt) {
                dA = fmaf(lm[tt][tid], zt[tt][tid], dA);
                dh1 += lm[tt][tid];
            }
        }
        if (lok) {
            for (int tt = 0; tt < SHG_TT; ++tt) {
                const long row = row0 + tt;
                if (row >= total) break;
                const bool m = (masks[(size_t)row * LW + (l >> 5)] >> (l & 31)) & 1u;
                float u = h2l, d = 0.f;
#pragma unroll
                for (int k = 0; k < MP; ++k) {
                    u = fmaf(w2r[k], zt[tt][k], u);
                    d = fmaf(w1c[k], lm[tt][k], d);
                }
                const float ru = m ? u : 0.f;
                d = m ? d : 0.f;
                dh2 += d;
#pragma unroll
                for (int k = 0; k < MP; ++k) {
                    dW1c[k] = fmaf(lm[tt][k], ru, dW1c[k]);
                    dW2r[k] = fmaf(d, zt[tt][k], dW2r[k]);
                }
            }
        }
    }
    const size_t stride = (size_t)2 * M * L + L + 2 * M;
    float *pp = part + (size_t)blockIdx.x * stride;
    if (lok) {
#pragma unroll
        for (int k = 0; k < MP; ++k)
            if (k < M) {
                pp[(size_t)k * L + l] = dW1c[k];
                pp[(size_t)M * L + (size_t)l * M + k] = dW2r[k];
            }
        pp[(size_t)2 * M * L + l] = dh2;
    }
    if (own_latent) {
        pp[(size_t)2 * M * L + L + tid] = dA;
        pp[(size_t)2 * M * L + L + M + tid] = dh1;
    }
}

// float64 sum over nrows partial rows of length width, then scattered to the outputs
__global__ void k_reduce_rows(const float *__restrict__ part, int nrows, int width, int M, int L,
                              float *__restrict__ dW1, float *__restrict__ dW2, float *__restrict__ dh2,
                              float *__restrict__ dA, float *__restrict__ dh1) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= width) return;
    double s0 = 0.0, s1 = 0.0;
    int r = 0;
    for (; r + 1 < nrows; r += 2) {
        s0 += (double)part[(size_t)r * width + e];
        s1 += (double)part[(size_t)(r + 1) * width + e];
    }
    if (r < nrows) s0 += (double)part[(size_t)r * width + e];
    const float v = (float)(s0 + s1);
    const int ML = M * L;
    if (e < ML) {
        if (dW1) dW1[e] = v;
    } else if (e < 2 * ML) {
        if (dW2) dW2[e - ML] = v;
    } else if (e < 2 * ML + L) {
        if (dh2) dh2[e - 2 * ML] = v;
    } else if (e < 2 * ML + L + M) {
        if (dA) dA[e - 2 * ML - L] = v;
    } else {
        if (dh1) dh1[e - 2 * ML - L - M] = v;
    }
}

// MSE seed g_t = scale * [z_t[:N] - x_t; 0] (used by the stored-Jacobian adjoint)
__global__ void k_mse_seed(const float *__restrict__ z, const float *__restrict__ x, float scale, int B, int T, int M,
                           int N, float *__restrict__ g) {
    const size_t n = (size_t)B * T * M;
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n; e += (size_t)gridDim.x * blockDim.x) {
        const int i = (int)(e % M);
        const size_t bt = e / M;
        const int b = (int)(bt / T), s = (int)(bt % T);
        g[e] = i < N ? scale * (z[e] - x[((size_t)b * (T + 1) + s + 1) * N + i]) : 0.f;
    }
}

// ---------------------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------------------
size_t sh_resjac_lds(int M, int L) {
    const int MP = padded_dim(M), LQ = sh_LQ(L);
    return (size_t)(SH_TT * MP + SH_TT * LQ + MP * LQ + 4 * (MP / 16) * 64 * 4) * sizeof(float);
}

static int sh_LP(int L) { return (L + 15) / 16 * 16; }

size_t sh_jacform_lds(int M, int L) { return (size_t)2 * padded_dim(M) * sh_LP(L) * sizeof(float); }

int launch_resjac_shplrnn(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *F, float *r,
                          uint32_t *masks, const int *active, hipStream_t st) {
    const long ntiles = ((long)a.B * a.T + SH_TT - 1) / SH_TT;
    const int grid = (int)(ntiles < 4096 ? ntiles : 4096);
    const size_t lds = sh_resjac_lds(a.M, a.L);
    KTimer kt("k_resjac_shplrnn", st);
    const int MP = padded_dim(a.M);
#define RS(MPV) \
    hipLaunchKernelGGL(k_resjac_shplrnn<MPV>, dim3(grid), dim3(256), lds, st, a, z, zalt, zsel, F, r, masks, active)
    if (MP == 16) RS(16); else if (MP == 32) RS(32); else RS(64);
#undef RS
    DEER_LAUNCH_CHECK("k_resjac_shplrnn");
    return DEER_OK;
}

int launch_jacform_shplrnn(const ShArgs &a, const uint32_t *masks, float *J, const int *active, const float *gamma,
                           hipStream_t st) {
    const int MP = padded_dim(a.M);
    const int LP = sh_LP(a.L);
    const size_t lds = sh_jacform_lds(a.M, a.L);
    const long total = (long)a.B * a.T;
    KTimer kt("k_jacform_shplrnn", st);
#define JF(MPV, NTV)                                                                                              \
    {                                                                                                             \
        const long groups = (total + NTV - 1) / NTV;                                                              \
        const long want = (groups + 3) / 4;                                                                       \
        const int grid = (int)(want < 2048 ? want : 2048);                                                        \
        hipLaunchKernelGGL((k_jacform_shplrnn<MPV, NTV>), dim3(grid), dim3(256), lds, st, a, masks, J, active, gamma, \
                           LP);                                                                              \
    }
    if (MP == 16) JF(16, 4) else if (MP == 32) JF(32, 4) else JF(64, 1)
#undef JF
    DEER_LAUNCH_CHECK("k_jacform_shplrnn");
    return DEER_OK;
}

size_t sh_grads_part_floats(int M, int L, int *nblocks) {
    *nblocks = 512;
    return (size_t)(*nblocks) * ((size_t)2 * M * L + L + 2 * M);
}

int launch_grads_shplrnn(const ShArgs &a, const float *z, const float *lam, const uint32_t *masks, float *part,
                         const deer_grads *gr, hipStream_t st) {
    int nb = 0;
    sh_grads_part_floats(a.M, a.L, &nb);
    const int MP = padded_dim(a.M);
    const dim3 grid(nb, (a.L + SHG_THREADS - 1) / SHG_THREADS);
    {
        KTimer kt("k_grads_shplrnn", st);
        if (MP == 16) hipLaunchKernelGGL(k_grads_shplrnn<16>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        else if (MP == 32) hipLaunchKernelGGL(k_grads_shplrnn<32>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        else hipLaunchKernelGGL(k_grads_shplrnn<64>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        DEER_LAUNCH_CHECK("k_grads_shplrnn");
    }
    const int width = 2 * a.M * a.L + a.L + 2 * a.M;
    {
        KTimer kt("k_reduce_rows", st);
        hipLaunchKernelGGL(k_reduce_rows, dim3((width + 255) / 256), dim3(256), 0, st, part, nb, width, a.M, a.L, gr->W,
                           gr->W2, gr->h2, gr->A, gr->h);
        DEER_LAUNCH_CHECK("k_reduce_rows");
    }
    return DEER_OK;
}

int launch_mse_seed(const float *z, const float *x, float scale, int B, int T, int M, int N, float *g, hipStream_t st) {
    const size_t n = (size_t)B * T * M;
    const int grid = (int)((n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536);
    KTimer kt("k_mse_seed", st);
    hipLaunchKernelGGL(k_mse_seed, dim3(grid), dim3(256), 0, st, z, x, scale, B, T, M, N, g);
    DEER_LAUNCH_CHECK("k_mse_seed");
    return DEER_OK;
}

}  // namespace deer
