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
// over tiles; the inputs of the next tile are loaded into registers while a tile is
// processed.  The hidden pre-activations u = W2 z~ + h2 that decide the masks are summed on
// the VALU in a fixed order (left to right from h2, a rounding after every multiply and add),
// thread j holding W2 row j and the TT sums of hidden unit j, the TT values z~_k read from LDS
// as four 16-byte broadcasts per k; F = A z~ + W1 relu(u) + h1 is a [M x L] x [L x TT]
// product on the matrix cores with the k range split over the 4 waves, and the partial tiles
// are summed by the threads that loaded those four latents of the row (and keep z for r).
// dynamic LDS: z~^T[MP][TT] | ru[TT][LQ] | W1[MP][LQ] | partial F [4][NI][64][4]
// (LQ = L rounded up to 16, + 4 so that rows stay 16-byte aligned and spread over banks)
// ---------------------------------------------------------------------------------------
constexpr int SH_TT = 16;

static __host__ __device__ inline int sh_LQ(int L) { return (L + 15) / 16 * 16 + 4; }

template <int MP>
__global__ __launch_bounds__(256) void k_resjac_shplrnn(const ShArgs a, const float *zbuf, const float *zalt,
                                                        const int *__restrict__ zsel, float *__restrict__ F_out,
                                                        float *__restrict__ r_out, uint32_t *__restrict__ masks,
                                                        const int *__restrict__ active) {
    constexpr int NI = MP / 16, TT = SH_TT, NT4 = TT * MP / 4;   // threads owning 4 latents of a row
    static_assert(NT4 <= 256 && TT == 16, "tile shape");
    extern __shared__ __align__(16) float smem[];
    const int M = a.M, L = a.L, T = a.T, N = a.N, LQ = sh_LQ(L);
    float *zT = smem;                    // [MP][TT]  z~ transposed
    float *ru = zT + MP * TT;            // [TT][LQ], zero padded
    float *w1s = ru + TT * LQ;           // [MP][LQ] = W1, zero padded
    v4f *red = reinterpret_cast<v4f *>(w1s + MP * LQ);   // [4][NI][64]
    __shared__ int rowok[SH_TT];         // row of the tile exists and its sequence is active
    const int tid = threadIdx.x;
    const int lane = tid & 63, wv = tid >> 6, g = lane >> 4, c = lane & 15;
    const int LW = (L + 31) / 32;
    const float p = __fsub_rn(1.0f, a.alpha);
    for (int e = tid; e < MP * LQ; e += 256) {
        const int i = e / LQ, l = e % LQ;
        w1s[e] = (i < M && l < L) ? a.W1[i * L + l] : 0.f;
    }
    for (int e = tid; e < TT * LQ; e += 256) ru[e] = 0.f;
    const long total = (long)a.B * T;
    const long ntiles = (total + TT - 1) / TT;
    const int njg = (L + 15) / 16;
    // the tile's inputs owned by this thread (tid < NT4): latents i0..i0+3 of row rc, the same
    // elements whose residual it writes at the end of the tile
    const int rc = tid / (MP / 4), i0 = 4 * (tid % (MP / 4));
    float pz[4], px[4], pc[4], cz[4];   // z_{s-1} (or the initial state at s = 0), x_s, z_s
    bool plater = false;                // the fetched row exists and has s > 0
    bool pwarm = false;                 // ... and is a latent warm-up step (s <= tw: z~ = x)
    auto fetch = [&](long tile) {
        const long row = tile * TT + rc;
        const bool ok = tid < NT4 && tile < ntiles && row < total;
        int b = 0, s = 0;
        if (ok) row_at(row_base(tile * TT, T), rc, T, b, s);
        plater = ok && s > 0;
        pwarm = plater && s <= a.tw;
        const float *z = cur_iter(zbuf, zalt, zsel, b);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = i0 + r;
            pz[r] = 0.f;
            px[r] = 0.f;
            pc[r] = 0.f;
            if (ok && i < M) {
                if (s == 0) {
                    pz[r] = a.z0 ? a.z0[(size_t)b * M + i] : (i < N ? a.x[(size_t)b * (T + 1) * N + i] : 0.f);
                } else if (a.zt) {
                    pz[r] = a.zt[((size_t)b * T + s) * M + i];   // the forced input itself (N = 0)
                } else {
                    pz[r] = z[((size_t)b * T + s - 1) * M + i];
                    if (i < N) px[r] = a.x[((size_t)b * (T + 1) + s) * N + i];
                }
                pc[r] = z[((size_t)b * T + s) * M + i];
            }
        }
    };
    // W2 rows of this thread's hidden units stay in registers when L <= 256
    float w2r[MP];
    float h2j = 0.f;
    auto load_w2 = [&](int j) {
        const bool jok = j < L;
#pragma unroll
        for (int k = 0; k < MP; ++k) w2r[k] = (jok && k < M) ? a.W2[(size_t)j * M + k] : 0.f;
        h2j = (jok && a.h2) ? a.h2[j] : 0.f;
    };
    if (L <= 256) load_w2(tid);
    long tile = blockIdx.x;
    fetch(tile);
    for (; tile < ntiles; tile += gridDim.x) {
        const long row0 = tile * TT;
        __syncthreads();   // the previous tile is done with zT, zc, ru and red
        if (tid < NT4) {
            const bool later = plater, warm = pwarm;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = i0 + r;
                float zt = pz[r];
                if (later && i < N) zt = warm ? px[r] : __fadd_rn(__fmul_rn(p, pz[r]), __fmul_rn(a.alpha, px[r]));
                zT[i * TT + rc] = zt;
                cz[r] = pc[r];
            }
        }
        if (tid < TT) {
            const long row = row0 + tid;
            int b = 0, sr = 0;
            if (row < total) row_at(row_base(row0, T), tid, T, b, sr);
            rowok[tid] = row < total && (!active || active[b]);
        }
        fetch(tile + gridDim.x);
        __syncthreads();
        // hidden pre-activations: left to right in k from h2, separate roundings.  The zero
        // padding adds exact zeros, so the value is the one of the unpadded sum.
        for (int jb = 0; jb < L; jb += 256) {
            const int j = jb + tid;
            const bool jok = j < L;
            if (L > 256) load_w2(j);
            float u[TT];
#pragma unroll
            for (int t = 0; t < TT; ++t) u[t] = h2j;
#pragma unroll
            for (int k = 0; k < MP; ++k) {
                const float4 *z4 = reinterpret_cast<const float4 *>(zT + k * TT);
#pragma unroll
                for (int t4 = 0; t4 < TT / 4; ++t4) {
                    const float4 v = z4[t4];
                    u[4 * t4] = __fadd_rn(u[4 * t4], __fmul_rn(w2r[k], v.x));
                    u[4 * t4 + 1] = __fadd_rn(u[4 * t4 + 1], __fmul_rn(w2r[k], v.y));
                    u[4 * t4 + 2] = __fadd_rn(u[4 * t4 + 2], __fmul_rn(w2r[k], v.z));
                    u[4 * t4 + 3] = __fadd_rn(u[4 * t4 + 3], __fmul_rn(w2r[k], v.w));
                }
            }
#pragma unroll
            for (int t = 0; t < TT; ++t)
                if (jok) ru[t * LQ + j] = u[t] > 0.f ? u[t] : 0.f;
        }
        __syncthreads();
        // mask words from relu(u) > 0 (= u > 0), rows of active sequences only
        if (masks) {
            for (int jb = 0; jb < L; jb += 256) {
                const int j = jb + tid;
                const int word = j / 32;
#pragma unroll 4
                for (int t = 0; t < TT; ++t) {
                    const uint64_t bal = __ballot(j < L && ru[t * LQ + j] > 0.f);
                    if (rowok[t] && (lane == 0 || lane == 32) && word < LW)
                        masks[(size_t)(row0 + t) * LW + word] = (uint32_t)(bal >> lane);
                }
            }
        }
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
        // four latents i0..i0+3 of row rc per thread: the four waves' partial sums of that
        // group are one 16-byte LDS entry each
        if (tid < NT4) {
            const int I = i0 / 16, gg = (i0 % 16) / 4;
            const long row = row0 + rc;
            const bool rok = rowok[rc] && i0 < M;
            if (rok) {
                v4f sum = red[I * 64 + 16 * gg + rc];
#pragma unroll
                for (int w = 1; w < 4; ++w) {
                    const v4f o = red[(w * NI + I) * 64 + 16 * gg + rc];
                    sum[0] += o[0]; sum[1] += o[1]; sum[2] += o[2]; sum[3] += o[3];
                }
                float Fv[4], rv[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = i0 + r;
                    Fv[r] = 0.f;
                    rv[r] = 0.f;
                    if (i < M) {
                        Fv[r] = fmaf(a.A[i], zT[i * TT + rc], sum[r]) + (a.h1 ? a.h1[i] : 0.f);
                        rv[r] = cz[r] - Fv[r];
                    }
                }
                const size_t e2 = (size_t)row * M + i0;
                if ((M & 3) == 0) {
                    if (F_out) *reinterpret_cast<float4 *>(F_out + e2) = make_float4(Fv[0], Fv[1], Fv[2], Fv[3]);
                    if (r_out) *reinterpret_cast<float4 *>(r_out + e2) = make_float4(rv[0], rv[1], rv[2], rv[3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (i0 + r < M) {
                            if (F_out) F_out[e2 + r] = Fv[r];
                            if (r_out) r_out[e2 + r] = rv[r];
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
    // rows (b, s) with t_lo <= s < t_hi, numbered b * len + (s - t_lo)
    const int t_lo = a.t_hi > a.t_lo ? a.t_lo : 0;
    const int len = a.t_hi > a.t_lo ? a.t_hi - a.t_lo : T;
    const long total = (long)a.B * len;
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
        long grow[NT];   // global row b * T + s of each of the NT rows
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const long row = row0 + nt;
            const long b = row / len;
            grow[nt] = b * T + t_lo + (row - b * len);
            rok[nt] = row < total && (!active || active[b]);
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
                const uint32_t w = masks[(size_t)grow[nt] * LW + word];
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
            float *Jp = Jout + (size_t)grow[nt] * M * M;
            // damping of the linearisation of this sequence (1 = exact Newton)
            const float gm = gamma ? gamma[grow[nt] / T] : 1.f;
#pragma unroll
            for (int I = 0; I < NI; ++I)
#pragma unroll
                for (int Jt = 0; Jt < NI; ++Jt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = 16 * I + 4 * g + r, col = 16 * Jt + c;
                        if (row < M && col < M) {
                            const float d = a.Cd ? a.Cd[row * M + col] : (row == col ? dI[I][r] : 0.f);
                            Jp[row * M + col] = gm * (acc[nt][I][Jt][r] + d);
                        }
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
                vz = (a.zt && s > 0) ? a.zt[(size_t)row * M + i]
                                     : forced_state(a.x, a.z0, z, b, s, i, T, M, a.N, a.alpha, a.tw);
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
// Column sums of part[nrows][width] in float64.  Block = 64 columns x RR_G row groups: thread
// (g, column) adds rows g, g + RR_G, ... (8 loads issued before their adds), then the row groups
// are added through LDS in a fixed order, so the sums do not depend on the launch.
constexpr int RR_G = 16;

__global__ __launch_bounds__(64 * RR_G) void k_reduce_rows(const float *__restrict__ part, int nrows, int width, int M,
                                                           int L, float *__restrict__ dW1, float *__restrict__ dW2,
                                                           float *__restrict__ dh2, float *__restrict__ dA,
                                                           float *__restrict__ dh1) {
    __shared__ double red[RR_G][64];
    const int col = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int e = blockIdx.x * 64 + col;
    const bool ok = e < width;
    double s = 0.0;
    for (int r0 = g; r0 < nrows; r0 += 8 * RR_G) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int r = r0 + k * RR_G;
            v[k] = (ok && r < nrows) ? part[(size_t)r * width + e] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) s += (double)v[k];
    }
    red[g][col] = s;
    __syncthreads();
    if (g != 0 || !ok) return;
    double t = red[0][col];
    for (int k = 1; k < RR_G; ++k) t += red[k][col];
    const float v = (float)t;
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

// MSE seed g_t = scale * [z_t[:N] - x_t; 0] (used by the stored-Jacobian adjoint); rows s < tw
// (the latent warm-up's states z_1..z_tw) are left out of the loss
__global__ void k_mse_seed(const float *__restrict__ z, const float *__restrict__ x, float scale, int B, int T, int M,
                           int N, float *__restrict__ g, int tw) {
    const size_t n = (size_t)B * T * M;
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n; e += (size_t)gridDim.x * blockDim.x) {
        const int i = (int)(e % M);
        const size_t bt = e / M;
        const int b = (int)(bt / T), s = (int)(bt % T);
        g[e] = (i < N && s >= tw) ? scale * (z[e] - x[((size_t)b * (T + 1) + s + 1) * N + i]) : 0.f;
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
    if (padded_dim(a.M) == 128) return launch_resjac_big(a, z, zalt, zsel, F, r, masks, active, st);
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
    if (padded_dim(a.M) == 128) return launch_jacform_big(a, masks, J, active, gamma, st);
    const int MP = padded_dim(a.M);
    const int LP = sh_LP(a.L);
    const size_t lds = sh_jacform_lds(a.M, a.L);
    const long total = (long)a.B * (a.t_hi > a.t_lo ? a.t_hi - a.t_lo : a.T);
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
    if (MP == 128) {
        int rc = launch_grads_big(a, z, lam, masks, part, nb, st);
        if (rc) return rc;
    } else {
        KTimer kt("k_grads_shplrnn", st);
        if (MP == 16) hipLaunchKernelGGL(k_grads_shplrnn<16>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        else if (MP == 32) hipLaunchKernelGGL(k_grads_shplrnn<32>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        else hipLaunchKernelGGL(k_grads_shplrnn<64>, grid, dim3(SHG_THREADS), 0, st, a, z, lam, masks, part);
        DEER_LAUNCH_CHECK("k_grads_shplrnn");
    }
    const int width = 2 * a.M * a.L + a.L + 2 * a.M;
    {
        KTimer kt("k_reduce_rows", st);
        hipLaunchKernelGGL(k_reduce_rows, dim3((width + 63) / 64), dim3(64 * RR_G), 0, st, part, nb, width, a.M, a.L,
                           gr->W, gr->W2, gr->h2, gr->A, gr->h);
        DEER_LAUNCH_CHECK("k_reduce_rows");
    }
    return DEER_OK;
}

int launch_mse_seed(const float *z, const float *x, float scale, int B, int T, int M, int N, float *g, hipStream_t st,
                    int tw) {
    const size_t n = (size_t)B * T * M;
    const int grid = (int)((n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536);
    KTimer kt("k_mse_seed", st);
    hipLaunchKernelGGL(k_mse_seed, dim3(grid), dim3(256), 0, st, z, x, scale, B, T, M, N, g, tw);
    DEER_LAUNCH_CHECK("k_mse_seed");
    return DEER_OK;
}

}  // namespace deer
