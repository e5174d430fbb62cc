// One-launch GTF-DEER solve for small vanilla PLRNNs (M <= 4, T <= 4096, a fixed number of
// plain Newton updates: Alg. GTF-DEER with the update count given, eq. GTF_DEER_update).
// One workgroup per sequence runs every update: each thread takes one chunk of the sequence and
// forms its affine map (the product of the chunk's forced Jacobians and its local solution) in
// registers, the carries across chunks go through LDS in two levels (group maps composed in
// parallel, a walk over the groups, every group re-walked), and each chunk is re-walked from
// its carry with the update written in place.  At these sizes a pass of the general path is
// bound by latency and launches (three kernels per update); here the whole solve is one launch.
#include "common.h"
#include "launch.h"

namespace deer {

namespace {
constexpr int SMS = 4;     // padded latent dimension
constexpr int SNT = 512;   // threads = chunks per workgroup
constexpr int SNG = 16;    // carry groups
constexpr int SPV = SMS * SMS + SMS;
constexpr int SC = 8;      // steps per chunk (T <= SNT * SC)
}  // namespace

__global__ __launch_bounds__(SNT) void k_newton_small(const float *__restrict__ A, const float *__restrict__ W,
                                                      const float *__restrict__ h, float alpha, int N,
                                                      const float *__restrict__ x, const float *__restrict__ z0,
                                                      float *__restrict__ z, int T, int M, int nc, int iters,
                                                      uint32_t *__restrict__ norm_bits) {
    __shared__ float Pm[SNT][SPV];    // chunk maps: P (row-major) then v
    __shared__ float Gm[SNG][SPV];    // group maps
    __shared__ float Xg[SNG][SMS];    // carry entering every group
    __shared__ float Xc[SNT][SMS];    // carry entering every chunk
    __shared__ uint32_t red[SNT / 64];
    const int b = blockIdx.x, c = threadIdx.x;
    float Ai[SMS], hi[SMS], pj[SMS], Wm[SMS][SMS];
#pragma unroll
    for (int i = 0; i < SMS; ++i) {
        Ai[i] = i < M ? A[i] : 0.f;
        hi[i] = (h && i < M) ? h[i] : 0.f;
        pj[i] = i < N ? __fsub_rn(1.0f, alpha) : 1.0f;
#pragma unroll
        for (int j = 0; j < SMS; ++j) Wm[i][j] = (i < M && j < M) ? W[i * M + j] : 0.f;
    }
    const float *xb = x + (size_t)b * (T + 1) * N;
    float *zb = z + (size_t)b * T * M;
    const bool act = c < nc;
    const int s0 = c * SC, s1 = act ? min(s0 + SC, T) : s0;
    // the chunk's data rows x_s (forced latents) stay in registers for the whole solve, its
    // iterate rows are loaded once per update (both phases use the same, not yet updated, z)
    float xr[SC][SMS], zr[SC][SMS];
#pragma unroll
    for (int k = 0; k < SC; ++k)
#pragma unroll
        for (int i = 0; i < SMS; ++i) xr[k][i] = (s0 + k < s1 && i < N) ? xb[(size_t)(s0 + k) * N + i] : 0.f;
    float zinit[SMS];
#pragma unroll
    for (int i = 0; i < SMS; ++i)
        zinit[i] = i >= M ? 0.f : (z0 ? z0[(size_t)b * M + i] : (i < N ? xb[i] : 0.f));

    // forced input of step s = s0 + k (array index) from z_{s-1}, then F and J~ = J_F P_alpha
    auto lin = [&](int k, const float *zp, float *F, float (*J)[SMS]) {
        float zt[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            if (s0 + k == 0) zt[i] = zinit[i];
            else if (i < N) zt[i] = __fadd_rn(__fmul_rn(pj[i], zp[i]), __fmul_rn(alpha, xr[k][i]));
            else zt[i] = zp[i];
        }
        float rl[SMS];
#pragma unroll
        for (int j = 0; j < SMS; ++j) rl[j] = zt[j] > 0.f ? zt[j] : 0.f;
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < SMS; ++j) a = fmaf(Wm[i][j], rl[j], a);
            F[i] = fmaf(Ai[i], zt[i], a) + hi[i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) {
                const float dj = (i == j ? Ai[i] : 0.f) + (zt[j] > 0.f ? Wm[i][j] : 0.f);
                J[i][j] = dj * pj[j];
            }
        }
    };
    auto load_row = [&](int s, float *v) {
#pragma unroll
        for (int i = 0; i < SMS; ++i) v[i] = i < M ? zb[(size_t)s * M + i] : 0.f;
    };
    // y <- P y + v for a map stored row-major with v after it
    auto apply = [&](const float *map, float *y) {
        float t[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            float a = map[SMS * SMS + i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) a = fmaf(map[i * SMS + j], y[j], a);
            t[i] = a;
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) y[i] = t[i];
    };

    uint32_t emax = 0u;
    for (int it = 0; it < iters; ++it) {
        // z_{s0-1} of this iterate, read before any thread writes the update of this pass
        float zbnd[SMS];
        if (act && s0 > 0) load_row(s0 - 1, zbnd);
        else {
#pragma unroll
            for (int i = 0; i < SMS; ++i) zbnd[i] = 0.f;
        }
#pragma unroll
        for (int k = 0; k < SC; ++k)
#pragma unroll
            for (int i = 0; i < SMS; ++i) zr[k][i] = (s0 + k < s1 && i < M) ? zb[(size_t)(s0 + k) * M + i] : 0.f;
        // chunk map: P = J~_{s1-1} ... J~_{s0}, v = Delta_{s1-1} from a zero carry
        float P[SMS][SMS], v[SMS], zp[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            v[i] = 0.f;
            zp[i] = zbnd[i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) P[i][j] = i == j ? 1.f : 0.f;
        }
#pragma unroll
        for (int k = 0; k < SC; ++k) {
            if (s0 + k >= s1) break;
            float F[SMS], J[SMS][SMS];
            const float *zs = zr[k];
            lin(k, zp, F, J);
            float Pn[SMS][SMS], vn[SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                float a = zs[i] - F[i];
                a = -a;
#pragma unroll
                for (int k = 0; k < SMS; ++k) a = fmaf(J[i][k], v[k], a);
                vn[i] = a;
#pragma unroll
                for (int j = 0; j < SMS; ++j) {
                    float q = 0.f;
#pragma unroll
                    for (int k = 0; k < SMS; ++k) q = fmaf(J[i][k], P[k][j], q);
                    Pn[i][j] = q;
                }
            }
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                v[i] = vn[i];
                zp[i] = zs[i];
#pragma unroll
                for (int j = 0; j < SMS; ++j) P[i][j] = Pn[i][j];
            }
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            Pm[c][SMS * SMS + i] = v[i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) Pm[c][i * SMS + j] = P[i][j];
        }
        __syncthreads();
        // carries: group maps G = P_{k1-1} ... P_{k0} with their local solutions, in parallel
        const int GC = (nc + SNG - 1) / SNG;
        if (c < SNG) {
            float G[SMS][SMS], g[SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                g[i] = 0.f;
#pragma unroll
                for (int j = 0; j < SMS; ++j) G[i][j] = i == j ? 1.f : 0.f;
            }
            const int k0 = min(c * GC, nc), k1 = min(k0 + GC, nc);
            for (int k = k0; k < k1; ++k) {
                const float *pk = Pm[k];
                float Gn[SMS][SMS];
#pragma unroll
                for (int i = 0; i < SMS; ++i)
#pragma unroll
                    for (int j = 0; j < SMS; ++j) {
                        float q = 0.f;
#pragma unroll
                        for (int l = 0; l < SMS; ++l) q = fmaf(pk[i * SMS + l], G[l][j], q);
                        Gn[i][j] = q;
                    }
                apply(pk, g);
#pragma unroll
                for (int i = 0; i < SMS; ++i)
#pragma unroll
                    for (int j = 0; j < SMS; ++j) G[i][j] = Gn[i][j];
            }
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                Gm[c][SMS * SMS + i] = g[i];
#pragma unroll
                for (int j = 0; j < SMS; ++j) Gm[c][i * SMS + j] = G[i][j];
            }
        }
        __syncthreads();
        if (c == 0) {
            float X[SMS] = {0.f, 0.f, 0.f, 0.f};
            for (int g2 = 0; g2 < SNG; ++g2) {
#pragma unroll
                for (int i = 0; i < SMS; ++i) Xg[g2][i] = X[i];
                apply(Gm[g2], X);
            }
        }
        __syncthreads();
        if (c < SNG) {
            float X[SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i) X[i] = Xg[c][i];
            const int k0 = min(c * GC, nc), k1 = min(k0 + GC, nc);
            for (int k = k0; k < k1; ++k) {
#pragma unroll
                for (int i = 0; i < SMS; ++i) Xc[k][i] = X[i];
                apply(Pm[k], X);
            }
        }
        __syncthreads();
        // fix-up: Delta from the carry, the update written in place
        float D[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            D[i] = act ? Xc[c][i] : 0.f;
            zp[i] = zbnd[i];
        }
        const bool last = it == iters - 1;
#pragma unroll
        for (int k = 0; k < SC; ++k) {
            if (s0 + k >= s1) break;
            const int s = s0 + k;
            float F[SMS], J[SMS][SMS];
            const float *zs = zr[k];
            lin(k, zp, F, J);
            float Dn[SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                float a = -(zs[i] - F[i]);
#pragma unroll
                for (int k = 0; k < SMS; ++k) a = fmaf(J[i][k], D[k], a);
                Dn[i] = a;
            }
#pragma unroll
            for (int i = 0; i < SMS; ++i) {
                D[i] = Dn[i];
                if (i < M) {
                    zb[(size_t)s * M + i] = zs[i] + D[i];
                    if (last) {
                        const uint32_t ab = abs_bits(D[i]);
                        emax = emax > ab ? emax : ab;
                    }
                }
                zp[i] = zs[i];
            }
        }
        __syncthreads();
    }
    emax = wave_max_u32(emax);
    if ((c & 63) == 0) red[c >> 6] = emax;
    __syncthreads();
    if (c == 0) {
        uint32_t e = red[0];
#pragma unroll
        for (int w = 1; w < SNT / 64; ++w) e = e > red[w] ? e : red[w];
        norm_bits[b] = e;
    }
}

// The adjoint of the same small problems in one launch (gradients appendix: lam_{s} =
// J~_{s+1}^T lam_{s+1} + g_s from the end, eq. backward_recursion): every thread takes an
// 8-step chunk, forms the map of its chunk in reverse (the product of the transposed
// Jacobians and the local adjoint from a zero carry), the carries run over the chunks from
// the last one in two levels through LDS, and each chunk is re-walked from its carry with the
// adjoint (optionally) written and the parameter-gradient partial sums of the thread,
//   dW_ij += lam_i relu(z~_j), dA_i += lam_i z~_i, dh_i += lam_i,
// summed over the workgroup into gpart[b][SMS][SMS + 2] for the float64 reduction over the batch.
__global__ __launch_bounds__(SNT) void k_adjoint_small(const float *__restrict__ A, const float *__restrict__ W,
                                                       float alpha, int N, const float *__restrict__ x,
                                                       const float *__restrict__ z0, const float *__restrict__ z,
                                                       const float *__restrict__ g, float seed_scale, int T, int M,
                                                       int nc, float *__restrict__ lam, float *__restrict__ gpart,
                                                       float *__restrict__ dA, float *__restrict__ dW,
                                                       float *__restrict__ dh) {
    __shared__ float Pm[SNT][SPV];
    __shared__ float Gm[SNG][SPV];
    __shared__ float Xg[SNG][SMS];
    __shared__ float Xc[SNT][SMS];
    __shared__ float red[SNT / 64][SMS * (SMS + 2)];
    const int b = blockIdx.x, c = threadIdx.x;
    float Ai[SMS], pj[SMS], Wm[SMS][SMS];
#pragma unroll
    for (int i = 0; i < SMS; ++i) {
        Ai[i] = i < M ? A[i] : 0.f;
        pj[i] = i < N ? __fsub_rn(1.0f, alpha) : 1.0f;
#pragma unroll
        for (int j = 0; j < SMS; ++j) Wm[i][j] = (i < M && j < M) ? W[i * M + j] : 0.f;
    }
    const float *xb = x + (size_t)b * (T + 1) * N;
    const float *zb = z + (size_t)b * T * M;
    const bool act = c < nc;
    const int s0 = c * SC, s1 = act ? min(s0 + SC, T) : s0;
    // forced inputs z~_s for s = s0 .. s0 + SC (the last one feeds J~ of the chunk's last step)
    // and the cotangent rows g_s of the chunk
    float zt[SC + 1][SMS], gr[SC][SMS];
#pragma unroll
    for (int k = 0; k <= SC; ++k) {
        const int s = s0 + k;
        const bool ok = act && s < T && (k < SC || s < T);
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            float v = 0.f;
            if (ok && i < M) {
                if (s == 0) v = z0 ? z0[(size_t)b * M + i] : (i < N ? xb[i] : 0.f);
                else if (i < N) v = __fadd_rn(__fmul_rn(pj[i], zb[(size_t)(s - 1) * M + i]), __fmul_rn(alpha, xb[(size_t)s * N + i]));
                else v = zb[(size_t)(s - 1) * M + i];
            }
            zt[k][i] = v;
        }
    }
#pragma unroll
    for (int k = 0; k < SC; ++k) {
        const int s = s0 + k;
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            float v = 0.f;
            if (s < s1 && i < M) {
                if (g) v = g[((size_t)b * T + s) * M + i];
                else if (i < N) v = __fmul_rn(seed_scale, __fsub_rn(zb[(size_t)s * M + i], xb[(size_t)(s + 1) * N + i]));
            }
            gr[k][i] = v;
        }
    }
    // y <- J~_{s+1}^T y + g_s, J~_{s+1} = (diag(A) + W diag(m)) P_alpha at z~_{s+1}; J~_T = 0
    auto step_t = [&](int k, const float *y, float *out) {
        const bool has = s0 + k + 1 < T;
        const float *zn = zt[k + 1];
#pragma unroll
        for (int j = 0; j < SMS; ++j) {
            float a = gr[k][j];
            if (has) {
                // (J~^T y)_j = p_j (A_j y_j + m_j sum_i W_ij y_i)
                float wsum = 0.f;
#pragma unroll
                for (int i = 0; i < SMS; ++i) wsum = fmaf(Wm[i][j], y[i], wsum);
                const float t = fmaf(Ai[j], y[j], zn[j] > 0.f ? wsum : 0.f);
                a = fmaf(pj[j], t, a);
            }
            out[j] = a;
        }
    };
    // map P (row-major) and local adjoint v of the chunk: y_{s0} = P y_{s1} + v
    float P[SMS][SMS], v[SMS];
#pragma unroll
    for (int i = 0; i < SMS; ++i) {
        v[i] = 0.f;
#pragma unroll
        for (int j = 0; j < SMS; ++j) P[i][j] = i == j ? 1.f : 0.f;
    }
#pragma unroll
    for (int k = SC - 1; k >= 0; --k) {
        if (s0 + k >= s1) continue;
        float vn[SMS];
        step_t(k, v, vn);
        // P <- J~^T P: column by column, without the cotangent
        float Pn[SMS][SMS];
#pragma unroll
        for (int col = 0; col < SMS; ++col) {
            float y[SMS], o[SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i) y[i] = P[i][col];
            const bool has = s0 + k + 1 < T;
            const float *zn = zt[k + 1];
#pragma unroll
            for (int j = 0; j < SMS; ++j) {
                float wsum = 0.f;
#pragma unroll
                for (int i = 0; i < SMS; ++i) wsum = fmaf(Wm[i][j], y[i], wsum);
                o[j] = has ? pj[j] * fmaf(Ai[j], y[j], zn[j] > 0.f ? wsum : 0.f) : 0.f;
            }
#pragma unroll
            for (int j = 0; j < SMS; ++j) Pn[j][col] = o[j];
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            v[i] = vn[i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) P[i][j] = Pn[i][j];
        }
    }
#pragma unroll
    for (int i = 0; i < SMS; ++i) {
        Pm[c][SMS * SMS + i] = v[i];
#pragma unroll
        for (int j = 0; j < SMS; ++j) Pm[c][i * SMS + j] = P[i][j];
    }
    __syncthreads();
    // carries from the last chunk: X(nc - 1) = 0, X(k - 1) = P_k X(k) + v_k; processing index
    // l = nc - 1 - k, groups of GC in processing order
    auto apply = [&](const float *map, float *y) {
        float t[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            float a = map[SMS * SMS + i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) a = fmaf(map[i * SMS + j], y[j], a);
            t[i] = a;
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) y[i] = t[i];
    };
    const int GC = (nc + SNG - 1) / SNG;
    if (c < SNG) {
        float G[SMS][SMS], gv[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            gv[i] = 0.f;
#pragma unroll
            for (int j = 0; j < SMS; ++j) G[i][j] = i == j ? 1.f : 0.f;
        }
        const int l0 = min(c * GC, nc), l1 = min(l0 + GC, nc);
        for (int l = l0; l < l1; ++l) {
            const float *pk = Pm[nc - 1 - l];
            float Gn[SMS][SMS];
#pragma unroll
            for (int i = 0; i < SMS; ++i)
#pragma unroll
                for (int j = 0; j < SMS; ++j) {
                    float q = 0.f;
#pragma unroll
                    for (int k = 0; k < SMS; ++k) q = fmaf(pk[i * SMS + k], G[k][j], q);
                    Gn[i][j] = q;
                }
            apply(pk, gv);
#pragma unroll
            for (int i = 0; i < SMS; ++i)
#pragma unroll
                for (int j = 0; j < SMS; ++j) G[i][j] = Gn[i][j];
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
            Gm[c][SMS * SMS + i] = gv[i];
#pragma unroll
            for (int j = 0; j < SMS; ++j) Gm[c][i * SMS + j] = G[i][j];
        }
    }
    __syncthreads();
    if (c == 0) {
        float X[SMS] = {0.f, 0.f, 0.f, 0.f};
        for (int g2 = 0; g2 < SNG; ++g2) {
#pragma unroll
            for (int i = 0; i < SMS; ++i) Xg[g2][i] = X[i];
            apply(Gm[g2], X);
        }
    }
    __syncthreads();
    if (c < SNG) {
        float X[SMS];
#pragma unroll
        for (int i = 0; i < SMS; ++i) X[i] = Xg[c][i];
        const int l0 = min(c * GC, nc), l1 = min(l0 + GC, nc);
        for (int l = l0; l < l1; ++l) {
            const int k = nc - 1 - l;
#pragma unroll
            for (int i = 0; i < SMS; ++i) Xc[k][i] = X[i];
            apply(Pm[k], X);
        }
    }
    __syncthreads();
    // re-walk from the carry with the gradient partials
    float L[SMS], gw[SMS][SMS + 2];
#pragma unroll
    for (int i = 0; i < SMS; ++i) {
        L[i] = act ? Xc[c][i] : 0.f;
#pragma unroll
        for (int j = 0; j < SMS + 2; ++j) gw[i][j] = 0.f;
    }
#pragma unroll
    for (int k = SC - 1; k >= 0; --k) {
        if (s0 + k >= s1) continue;
        float Ln[SMS];
        step_t(k, L, Ln);
#pragma unroll
        for (int i = 0; i < SMS; ++i) L[i] = Ln[i];
        if (lam) {
#pragma unroll
            for (int i = 0; i < SMS; ++i)
                if (i < M) lam[((size_t)b * T + s0 + k) * M + i] = L[i];
        }
#pragma unroll
        for (int i = 0; i < SMS; ++i) {
#pragma unroll
            for (int j = 0; j < SMS; ++j) gw[i][j] = fmaf(L[i], zt[k][j] > 0.f ? zt[k][j] : 0.f, gw[i][j]);
            gw[i][SMS] = fmaf(L[i], zt[k][i], gw[i][SMS]);
            gw[i][SMS + 1] += L[i];
        }
    }
    // workgroup sum of the partials (waves, then the eight wave sums)
#pragma unroll
    for (int i = 0; i < SMS; ++i)
#pragma unroll
        for (int j = 0; j < SMS + 2; ++j) {
            float t = gw[i][j];
            for (int off = 32; off > 0; off >>= 1) t += __shfl_xor(t, off, 64);
            if ((c & 63) == 0) red[c >> 6][i * (SMS + 2) + j] = t;
        }
    __syncthreads();
    if (c < SMS * (SMS + 2)) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < SNT / 64; ++w) t += red[w][c];
        if (gpart) gpart[(size_t)b * SMS * (SMS + 2) + c] = t;
        // a single sequence: the gradients themselves, no reduction over the batch
        const int i = c / (SMS + 2), j = c % (SMS + 2);
        if (i < M && (j >= SMS || j < M)) {
            if (j < SMS) {
                if (dW) dW[i * M + j] = t;
            } else if (j == SMS) {
                if (dA) dA[i] = t;
            } else if (dh) {
                dh[i] = t;
            }
        }
    }
}

bool newton_small_fits(int M, int T, int fixed_iters) { return M <= SMS && T <= SNT * SC && fixed_iters > 0; }

int launch_newton_small(const PlrnnArgs &a, float *z, int iters, uint32_t *norm_bits, hipStream_t st) {
    if (a.tw > 0) {
        set_error("the one-launch solve takes no latent warm-up");
        return DEER_ERR_INVALID_ARG;
    }
    const int nc = (a.T + SC - 1) / SC;
    KTimer kt("k_newton_small", st);
    hipLaunchKernelGGL(k_newton_small, dim3(a.B), dim3(SNT), 0, st, a.A, a.W, a.h, a.alpha, a.N, a.x, a.z0, z, a.T, a.M,
                       nc, iters, norm_bits);
    DEER_LAUNCH_CHECK("k_newton_small");
    return DEER_OK;
}

}  // namespace deer

namespace deer {
bool adjoint_small_fits(int M, int T) { return M <= SMS && T <= SNT * SC; }

int launch_adjoint_small(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *lam,
                         float *gpart, float *dA, float *dW, float *dh, hipStream_t st) {
    if (a.tw > 0) {
        set_error("the one-launch adjoint takes no latent warm-up");
        return DEER_ERR_INVALID_ARG;
    }
    const int nc = (a.T + SC - 1) / SC;
    KTimer kt("k_adjoint_small", st);
    hipLaunchKernelGGL(k_adjoint_small, dim3(a.B), dim3(SNT), 0, st, a.A, a.W, a.alpha, a.N, a.x, a.z0, z, g,
                       seed_scale, a.T, a.M, nc, lam, gpart, dA, dW, dh);
    DEER_LAUNCH_CHECK("k_adjoint_small");
    return DEER_OK;
}
}  // namespace deer
