// General observation matrix B [N, M] of the linear read-out x^_t = B z_t (eq. shplrnn_nonlinear):
// the error-forcing projector P_alpha = I - alpha B^+ B and the forcing targets B^+ x_t (eq.
// error_forcing; Alg. GTF-DEER: pinv(B), P_alpha and P_1), the forced inputs of every step, the
// MSE seed of the read-out, and the gradient with respect to B (g_B of the IFT gradient).
//
//   k_obs_setup        one block: B^+ (Gauss-Jordan on the Gram matrix of the shorter side, float64),
//                      P_alpha, P_1, the Jacobian-formation operands W2 P and diag(A) P, in float32
//   k_obs_forced       z~_s = P_s z_s + alpha_s B^+ x_s for every step (P_1, alpha_s = 1 in the
//                      warm-up), z_0 = B^+ x_0 when no initial state is given; or the teacher
//                      states B^+ x_{s+1} (the initial Newton iterate)
//   k_obs_seed         g_t = scale B^T (B z_t - x_t) after the warm-up, 0 in it
//   k_obs_bgrad_part   per block float64 sums of mu z^T, mu x^T (mu = J_F(z~)^T lam) and
//                      (B z - x) z^T over its rows;  k_obs_bgrad_reduce sums the blocks
//   k_obs_bgrad_final  one block: g_B from the sums (differential of the pseudo-inverse)
#include "common.h"
#include "launch.h"

namespace deer {

constexpr int OBS_MAX = 64;   // M, N <= 64

__global__ __launch_bounds__(256) void k_obs_setup(ObsSetup s) {
    double *aug = s.aug;   // [K][2K] Gram matrix | identity (workspace; one block)
    __shared__ int piv_bad;
    const int N = s.N, M = s.M, L = s.L, tid = threadIdx.x;
    const bool wide = N <= M;                   // full row rank: B^+ = B^T (B B^T)^-1
    const int K = wide ? N : M, K2 = 2 * K;
    const float *Bf = s.B;
    auto Bv = [&](int n, int j) { return (double)Bf[(size_t)n * M + j]; };
    if (tid == 0) piv_bad = 0;
    for (int e = tid; e < K * K; e += 256) {
        const int i = e / K, j = e % K;
        double g = 0.0;
        if (wide)
            for (int k = 0; k < M; ++k) g += Bv(i, k) * Bv(j, k);
        else
            for (int k = 0; k < N; ++k) g += Bv(k, i) * Bv(k, j);
        aug[i * K2 + j] = g;
        aug[i * K2 + K + j] = i == j ? 1.0 : 0.0;
    }
    __syncthreads();
    double gmax = 0.0;
    for (int i = 0; i < K; ++i) gmax = fmax(gmax, fabs(aug[i * K2 + i]));
    // Gauss-Jordan with partial pivoting
    for (int c = 0; c < K; ++c) {
        __shared__ int prow;
        if (tid == 0) {
            int best = c;
            for (int r = c + 1; r < K; ++r)
                if (fabs(aug[r * K2 + c]) > fabs(aug[best * K2 + c])) best = r;
            prow = best;
            if (!(fabs(aug[best * K2 + c]) > 1e-13 * gmax)) piv_bad = 1;
        }
        __syncthreads();
        const int pr = prow;
        if (pr != c)
            for (int j = tid; j < K2; j += 256) {
                const double t = aug[c * K2 + j];
                aug[c * K2 + j] = aug[pr * K2 + j];
                aug[pr * K2 + j] = t;
            }
        __syncthreads();
        const double inv = 1.0 / aug[c * K2 + c];
        __syncthreads();
        for (int j = tid; j < K2; j += 256) aug[c * K2 + j] *= inv;
        __syncthreads();
        for (int e = tid; e < K * K2; e += 256) {
            const int r = e / K2, j = e % K2;
            if (r != c) {
                const double f = aug[r * K2 + c];
                if (j != c) aug[e] -= f * aug[c * K2 + j];
            }
        }
        __syncthreads();
        for (int r = tid; r < K; r += 256)
            if (r != c) aug[r * K2 + c] = 0.0;
        __syncthreads();
    }
    const double nan = __longlong_as_double(0x7ff8000000000000LL);
    const bool bad = piv_bad != 0;
    // B^+ [M][N]
    for (int e = tid; e < M * N; e += 256) {
        const int m = e / N, n = e % N;
        double v = 0.0;
        if (wide)
            for (int k = 0; k < N; ++k) v += Bv(k, m) * aug[k * K2 + K + n];
        else
            for (int k = 0; k < M; ++k) v += aug[m * K2 + K + k] * Bv(n, k);
        v = bad ? nan : v;
        s.Bp64[e] = v;
        s.Bp32[e] = (float)v;
    }
    for (int e = tid; e < N * M; e += 256) s.B64[e] = (double)Bf[e];
    __syncthreads();
    // P_1 = I - B^+ B and P_alpha = I - alpha B^+ B
    const double al = (double)s.alpha;
    for (int e = tid; e < M * M; e += 256) {
        const int i = e / M, j = e % M;
        double bb = 0.0;
        for (int n = 0; n < N; ++n) bb += s.Bp64[(size_t)i * N + n] * Bv(n, j);
        const double id = i == j ? 1.0 : 0.0;
        s.P164[e] = id - bb;
        s.P132[e] = (float)(id - bb);
        s.Pa32[e] = (float)(id - al * bb);
        const double a = (double)s.A[i];
        s.C1[e] = (float)(a * (id - bb));
        s.Ca[e] = (float)(a * (id - al * bb));
        s.Id[e] = (float)id;
    }
    __syncthreads();
    // W2 P for both projectors ([L][M]); the vanilla PLRNN takes W2 = I (then W2 P = P)
    for (int e = tid; e < L * M; e += 256) {
        const int l = e / M, j = e % M;
        double v1 = 0.0, va = 0.0;
        for (int k = 0; k < M; ++k) {
            const double w = s.W2 ? (double)s.W2[(size_t)l * M + k] : (l == k ? 1.0 : 0.0);
            const double bb = s.P164[(size_t)k * M + j];   // (I - B^+ B)[k][j]
            const double id = k == j ? 1.0 : 0.0;
            v1 += w * bb;
            va += w * (id - al * (id - bb));
        }
        s.V1[e] = (float)v1;
        s.Va[e] = (float)va;
    }
}

// One wave per row (b, s), lane i < M owns latent i.  mode 0: the forced input of step s + 1,
// zt[b, s] = P_s z_{s-1} + alpha_s B^+ x_s (s >= 1, z the current iterate; row s = 0 writes
// B^+ x_0 to z0e when no initial state is given).  mode 1: the teacher states
// out[b, s] = B^+ x_{s+1} (s = 0..T-1) and z0e as in mode 0.
__global__ __launch_bounds__(256) void k_obs_forced(int mode, const float *zbuf, const float *zalt,
                                                    const int *__restrict__ zsel, const float *__restrict__ x,
                                                    const float *__restrict__ z0, const float *__restrict__ Bp,
                                                    const float *__restrict__ Pa, const float *__restrict__ P1,
                                                    float alpha, int T_w, int B, int T, int M, int N,
                                                    float *__restrict__ out, float *__restrict__ z0e) {
    __shared__ float pa[OBS_MAX * OBS_MAX], p1[OBS_MAX * OBS_MAX], bp[OBS_MAX * OBS_MAX];
    __shared__ float zr[4][OBS_MAX], xr[4][OBS_MAX];
    const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63;
    for (int e = tid; e < M * M; e += 256) {
        pa[e] = Pa[e];
        p1[e] = P1[e];
    }
    for (int e = tid; e < M * N; e += 256) bp[e] = Bp[e];
    __syncthreads();
    const long rows = (long)B * T;
    for (long row0 = (long)blockIdx.x * 4; row0 < rows; row0 += (long)gridDim.x * 4) {
        const long row = row0 + wv;
        const bool ok = row < rows;
        const int b = ok ? (int)(row / T) : 0, s = ok ? (int)(row % T) : 0;
        // the x row this step needs: x_s (mode 0) or x_{s+1} (mode 1); z_{s-1} for mode 0
        const int xs = mode == 0 ? s : s + 1;
        const float *zc = cur_iter(zbuf, zalt, zsel, b);
        xr[wv][lane] = (ok && lane < N) ? x[((size_t)b * (T + 1) + xs) * N + lane] : 0.f;
        zr[wv][lane] = (ok && mode == 0 && s > 0 && lane < M) ? zc[((size_t)b * T + s - 1) * M + lane] : 0.f;
        __syncthreads();
        if (ok && lane < M) {
            float zb = 0.f;   // (B^+ x)_i
            for (int k = 0; k < N; ++k) zb = fmaf(bp[lane * N + k], xr[wv][k], zb);
            if (mode == 1) {
                out[((size_t)b * T + s) * M + lane] = zb;
            } else if (s > 0) {
                const bool warm = s <= T_w;
                const float *P = warm ? p1 : pa;
                const float as = warm ? 1.f : alpha;
                float v = 0.f;
                for (int j = 0; j < M; ++j) v = fmaf(P[lane * M + j], zr[wv][j], v);
                out[((size_t)b * T + s) * M + lane] = fmaf(as, zb, v);
            }
            if (s == 0 && !z0 && z0e) {
                float z00 = 0.f;   // B^+ x_0
                for (int k = 0; k < N; ++k) z00 = fmaf(bp[lane * N + k], x[((size_t)b * (T + 1)) * N + k], z00);
                z0e[(size_t)b * M + lane] = z00;
            }
        }
        __syncthreads();
    }
}

// g[b, s] = scale B^T (B z[b, s] - x[b, s + 1]) for s >= T_w, 0 for s < T_w; one wave per row
__global__ __launch_bounds__(256) void k_obs_seed(const float *__restrict__ z, const float *__restrict__ x,
                                                  const float *__restrict__ Bm, float scale, int T_w, int B, int T,
                                                  int M, int N, float *__restrict__ g) {
    __shared__ float bm[OBS_MAX * OBS_MAX];
    __shared__ float zr[4][OBS_MAX], er[4][OBS_MAX];
    const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63;
    for (int e = tid; e < N * M; e += 256) bm[e] = Bm[e];
    __syncthreads();
    const long rows = (long)B * T;
    for (long row0 = (long)blockIdx.x * 4; row0 < rows; row0 += (long)gridDim.x * 4) {
        const long row = row0 + wv;
        const bool ok = row < rows;
        const int b = ok ? (int)(row / T) : 0, s = ok ? (int)(row % T) : 0;
        zr[wv][lane] = (ok && lane < M) ? z[(size_t)row * M + lane] : 0.f;
        __syncthreads();
        if (ok && lane < N) {
            float e = 0.f;
            for (int j = 0; j < M; ++j) e = fmaf(bm[lane * M + j], zr[wv][j], e);
            er[wv][lane] = e - x[((size_t)b * (T + 1) + s + 1) * N + lane];
        }
        __syncthreads();
        if (ok && lane < M) {
            float v = 0.f;
            for (int n = 0; n < N; ++n) v = fmaf(bm[n * M + lane], er[wv][n], v);
            g[(size_t)row * M + lane] = s >= T_w ? scale * v : 0.f;
        }
        __syncthreads();
    }
}

// Per block float64 sums over its rows (b, s) of
//   S1 [M][M] += w_s mu_s z_{s-1}^T,   S2 [M][N] += w_s mu_s x_s^T   (s >= 1, w_s = alpha_s),
//   S2 += mu_0 x_0^T at s = 0 when z_0 = B^+ x_0 (no initial state given),
//   D  [N][M] += (B z_s - x_{s+1}) z_s^T for s >= T_w (the MSE's direct dependence on B),
// mu_s = J_F(z~_s)^T lam_s, with J_F [B,T,M,M] the unforced Jacobians.  The block walks its
// rows one at a time; each thread owns up to 16 entries of each sum.
constexpr int OBG_PER = 16;

__global__ __launch_bounds__(256) void k_obs_bgrad_part(const float *__restrict__ JF, const float *__restrict__ lam,
                                                        const float *__restrict__ z, const float *__restrict__ x,
                                                        const float *__restrict__ Bm, int z0_given, float alpha,
                                                        int T_w, int with_mse, int B, int T, int M, int N,
                                                        double *__restrict__ part) {
    __shared__ float mu[OBS_MAX], zp[OBS_MAX], zc[OBS_MAX], xs[OBS_MAX], er[OBS_MAX];
    __shared__ float bm[OBS_MAX * OBS_MAX];
    const int tid = threadIdx.x;
    for (int e = tid; e < N * M; e += 256) bm[e] = Bm[e];
    double s1[OBG_PER], s2[OBG_PER], dd[OBG_PER];
#pragma unroll
    for (int q = 0; q < OBG_PER; ++q) s1[q] = s2[q] = dd[q] = 0.0;
    const long rows = (long)B * T;
    const long per = (rows + gridDim.x - 1) / gridDim.x;
    const long r0 = (long)blockIdx.x * per, r1 = r0 + per < rows ? r0 + per : rows;
    __syncthreads();
    for (long row = r0; row < r1; ++row) {
        const int b = (int)(row / T), s = (int)(row % T);
        if (tid < M) {
            const float *Jr = JF + (size_t)row * M * M + tid;   // column tid of J_F
            const float *lr = lam + (size_t)row * M;
            float v = 0.f;
            for (int i = 0; i < M; ++i) v = fmaf(Jr[(size_t)i * M], lr[i], v);
            mu[tid] = v;
            zp[tid] = s > 0 ? z[(size_t)(row - 1) * M + tid] : 0.f;
            zc[tid] = z[(size_t)row * M + tid];
        }
        if (tid < N) xs[tid] = x[((size_t)b * (T + 1) + s) * N + tid];
        __syncthreads();
        if (tid < N) {
            float e = 0.f;
            for (int j = 0; j < M; ++j) e = fmaf(bm[tid * M + j], zc[j], e);
            er[tid] = e - x[((size_t)b * (T + 1) + s + 1) * N + tid];
        }
        __syncthreads();
        const double w = s == 0 ? (z0_given ? 0.0 : 1.0) : (s <= T_w ? 1.0 : (double)alpha);
        const bool use_d = with_mse && s >= T_w;
#pragma unroll
        for (int q = 0; q < OBG_PER; ++q) {
            const int e = tid + 256 * q;
            if (s > 0 && e < M * M) s1[q] += w * (double)mu[e / M] * (double)zp[e % M];
            if (w != 0.0 && e < M * N) s2[q] += w * (double)mu[e / N] * (double)xs[e % N];
            if (use_d && e < N * M) dd[q] += (double)er[e / M] * (double)zc[e % M];
        }
        __syncthreads();
    }
    const size_t S = (size_t)M * M + (size_t)M * N + (size_t)N * M;
    double *pp = part + (size_t)blockIdx.x * S;
#pragma unroll
    for (int q = 0; q < OBG_PER; ++q) {
        const int e = tid + 256 * q;
        if (e < M * M) pp[e] = s1[q];
        if (e < M * N) pp[(size_t)M * M + e] = s2[q];
        if (e < N * M) pp[(size_t)M * M + M * N + e] = dd[q];
    }
}

__global__ void k_obs_bgrad_reduce(const double *__restrict__ part, int nblk, int S, double *__restrict__ sum) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= S) return;
    double a = 0.0, c = 0.0;
    int r = 0;
    for (; r + 1 < nblk; r += 2) {
        a += part[(size_t)r * S + e];
        c += part[(size_t)(r + 1) * S + e];
    }
    if (r < nblk) a += part[(size_t)r * S + e];
    sum[e] = a + c;
}

// g_B = -B^+T (S1 P_1 + S2 B^+T) + (I - B B^+) E (B^+ B^+T) + (B^+T B^+) E P_1 + mse_scale D,
// E = S2^T - B S1^T: the sums of mu^T (dB^+) e - mu^T B^+ dB z over the forced inputs with
// dB^+ = -B^+ dB B^+ + B^+ B^+T dB^T (I - B B^+) + (I - B^+ B) dB^T B^+T B^+ (the differential
// of the pseudo-inverse at constant rank, Golub and Pereyra 1973).  One block, float64;
// t1 .. t4 are [64][64] float64 scratch matrices.
__global__ __launch_bounds__(256) void k_obs_bgrad_final(const double *__restrict__ sum, const double *__restrict__ Bp,
                                                         const double *__restrict__ Bm, const double *__restrict__ P1,
                                                         int M, int N, double mse_scale, double *__restrict__ t1,
                                                         double *__restrict__ t2, double *__restrict__ t3,
                                                         double *__restrict__ t4, float *__restrict__ gB) {
    const int tid = threadIdx.x;
    const double *S1 = sum, *S2 = sum + (size_t)M * M, *D = sum + (size_t)M * M + (size_t)M * N;
    // t1 [M][M] = S1 P_1 + S2 B^+T
    for (int e = tid; e < M * M; e += 256) {
        const int i = e / M, j = e % M;
        double v = 0.0;
        for (int k = 0; k < M; ++k) v += S1[i * M + k] * P1[k * M + j];
        for (int n = 0; n < N; ++n) v += S2[i * N + n] * Bp[j * N + n];
        t1[e] = v;
    }
    // t2 [N][M] = E = S2^T - B S1^T;  t3 [M][M] = B^+ B^+T;  t4 [N][N] = B^+T B^+
    for (int e = tid; e < N * M; e += 256) {
        const int n = e / M, j = e % M;
        double v = S2[j * N + n];
        for (int k = 0; k < M; ++k) v -= Bm[n * M + k] * S1[j * M + k];
        t2[e] = v;
    }
    for (int e = tid; e < M * M; e += 256) {
        const int i = e / M, j = e % M;
        double v = 0.0;
        for (int n = 0; n < N; ++n) v += Bp[i * N + n] * Bp[j * N + n];
        t3[e] = v;
    }
    for (int e = tid; e < N * N; e += 256) {
        const int a = e / N, c = e % N;
        double v = 0.0;
        for (int m = 0; m < M; ++m) v += Bp[m * N + a] * Bp[m * N + c];
        t4[e] = v;
    }
    __syncthreads();
    // g_B[n][j]
    for (int e = tid; e < N * M; e += 256) {
        const int n = e / M, j = e % M;
        double g = 0.0;
        for (int k = 0; k < M; ++k) g -= Bp[k * N + n] * t1[k * M + j];   // -B^+T t1
        // (I - B B^+) E B^+ B^+T:  (E t3)[a][j] summed with (I - B B^+)[n][a]
        for (int a = 0; a < N; ++a) {
            double bbp = a == n ? 1.0 : 0.0;   // (I - B B^+)[n][a]
            for (int m = 0; m < M; ++m) bbp -= Bm[n * M + m] * Bp[m * N + a];
            if (bbp == 0.0) continue;
            double et = 0.0;
            for (int k = 0; k < M; ++k) et += t2[a * M + k] * t3[k * M + j];
            g += bbp * et;
        }
        // B^+T B^+ E P_1
        for (int a = 0; a < N; ++a) {
            double ep = 0.0;
            for (int k = 0; k < M; ++k) ep += t2[a * M + k] * P1[k * M + j];
            g += t4[n * N + a] * ep;
        }
        g += mse_scale * D[n * M + j];
        gB[e] = (float)g;
    }
}

// ---- host launchers -------------------------------------------------------------------------

int launch_obs_setup(const ObsSetup &s, hipStream_t st) {
    KTimer kt("k_obs_setup", st);
    hipLaunchKernelGGL(k_obs_setup, dim3(1), dim3(256), 0, st, s);
    DEER_LAUNCH_CHECK("k_obs_setup");
    return DEER_OK;
}

static int obs_grid(long rows) {
    const long g = (rows + 3) / 4;
    return (int)(g < 4096 ? (g > 0 ? g : 1) : 4096);
}

int launch_obs_forced(int mode, const float *z, const float *zalt, const int *zsel, const float *x, const float *z0,
                      const float *Bp, const float *Pa, const float *P1, float alpha, int T_w, int B, int T, int M,
                      int N, float *out, float *z0e, hipStream_t st) {
    KTimer kt(mode == 1 ? "k_obs_teacher" : "k_obs_forced", st);
    hipLaunchKernelGGL(k_obs_forced, dim3(obs_grid((long)B * T)), dim3(256), 0, st, mode, z, zalt, zsel, x, z0, Bp,
                       Pa, P1, alpha, T_w, B, T, M, N, out, z0e);
    DEER_LAUNCH_CHECK("k_obs_forced");
    return DEER_OK;
}

int launch_obs_seed(const float *z, const float *x, const float *Bm, float scale, int T_w, int B, int T, int M, int N,
                    float *g, hipStream_t st) {
    KTimer kt("k_obs_seed", st);
    hipLaunchKernelGGL(k_obs_seed, dim3(obs_grid((long)B * T)), dim3(256), 0, st, z, x, Bm, scale, T_w, B, T, M, N, g);
    DEER_LAUNCH_CHECK("k_obs_seed");
    return DEER_OK;
}

constexpr int OBG_BLOCKS = 512;

size_t obs_bgrad_ws_doubles(int M, int N) {
    const size_t S = (size_t)M * M + 2 * (size_t)M * N;
    return (size_t)OBG_BLOCKS * S + S + 4 * (size_t)OBS_MAX * OBS_MAX;
}

int launch_obs_bgrad(const float *JF, const float *lam, const float *z, const float *x, const float *Bm32,
                     const double *Bp64, const double *Bm64, const double *P164, bool z0_given, float alpha, int T_w,
                     bool with_mse, double mse_scale, int B, int T, int M, int N, double *ws, float *gB,
                     hipStream_t st) {
    const int S = M * M + 2 * M * N;
    const long rows = (long)B * T;
    const int nblk = (int)(rows < OBG_BLOCKS ? rows : OBG_BLOCKS);
    double *part = ws, *sum = ws + (size_t)OBG_BLOCKS * S, *t = sum + S;
    {
        KTimer kt("k_obs_bgrad_part", st);
        hipLaunchKernelGGL(k_obs_bgrad_part, dim3(nblk), dim3(256), 0, st, JF, lam, z, x, Bm32, z0_given ? 1 : 0, alpha,
                           T_w, with_mse ? 1 : 0, B, T, M, N, part);
        DEER_LAUNCH_CHECK("k_obs_bgrad_part");
    }
    {
        KTimer kt("k_obs_bgrad_reduce", st);
        hipLaunchKernelGGL(k_obs_bgrad_reduce, dim3((S + 255) / 256), dim3(256), 0, st, part, nblk, S, sum);
        DEER_LAUNCH_CHECK("k_obs_bgrad_reduce");
    }
    {
        const size_t q = (size_t)OBS_MAX * OBS_MAX;
        KTimer kt("k_obs_bgrad_final", st);
        hipLaunchKernelGGL(k_obs_bgrad_final, dim3(1), dim3(256), 0, st, sum, Bp64, Bm64, P164, M, N, mse_scale, t,
                           t + q, t + 2 * q, t + 3 * q, gB);
        DEER_LAUNCH_CHECK("k_obs_bgrad_final");
    }
    return DEER_OK;
}

}  // namespace deer
