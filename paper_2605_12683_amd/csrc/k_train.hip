// The training step around the gradient (Alg. GTF-DEER, loop body after the solve): the MSE of
// the post-warm-up states (eq. mse_loss_warmup), the manifold attractor regularisation of the
// last M_r latents (eq. mar_loss_latent_initscale) added to the loss and to the gradient, and
// one Adam step on the parameters in place.  Parameters, gradients and the Adam moments share
// one layout: vanilla A [M] | W [M,M] | h [M]; shallow A [M] | W1 [M,L] | W2 [L,M] | h1 [M] | h2 [L].
#include "common.h"
#include "launch.h"

namespace deer {

namespace {
constexpr int TR_BLK = 256;
constexpr int TR_NB = 256;   // blocks of the loss partial sums

__device__ __forceinline__ double block_sum(double v, double *red) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    double t = 0.0;
    if (threadIdx.x == 0)
        for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w];
    return t;
}
}  // namespace

// partial sums of (z_t[i] - x_t[i])^2 over t > T_w, i < N (float64)
__global__ __launch_bounds__(TR_BLK) void k_mse_partial(const float *__restrict__ z, const float *__restrict__ x, int B,
                                                        int T, int M, int N, int T_w, double *__restrict__ part) {
    __shared__ double red[TR_BLK / 64];
    const long T2 = T - T_w, n = (long)B * T2 * N;
    double s = 0.0;
    for (long e = blockIdx.x * (long)TR_BLK + threadIdx.x; e < n; e += (long)gridDim.x * TR_BLK) {
        const long i = e % N, bt = e / N, t = bt % T2 + T_w, b = bt / T2;
        const double d = (double)z[(b * T + t) * M + i] - (double)x[(b * (T + 1) + t + 1) * N + i];
        s += d * d;
    }
    const double t = block_sum(s, red);
    if (threadIdx.x == 0) part[blockIdx.x] = t;
}

// MAR: the loss into mar[0] and its gradient added to g (one block)
__global__ __launch_bounds__(TR_BLK) void k_mar(int shallow, const float *__restrict__ A, const float *__restrict__ W,
                                                const float *__restrict__ V, const float *__restrict__ h, int M, int L,
                                                int M_r, float lam_mar, int p, float gamma_w, float gamma_v,
                                                float *__restrict__ g, double *__restrict__ mar) {
    __shared__ double red[TR_BLK / 64];
    const int i0 = M - M_r;
    const double c = (double)lam_mar / M_r;
    const int Lw = shallow ? L : M;
    float *gA = g, *gW = g + M;
    float *gV = shallow ? g + M + (size_t)M * L : nullptr;
    float *gh = shallow ? g + M + 2 * (size_t)M * L : g + M + (size_t)M * M;
    auto pen = [&](double u) { return p == 1 ? fabs(u) : u * u; };
    auto dpen = [&](double u) { return p == 1 ? (u > 0.0 ? 1.0 : (u < 0.0 ? -1.0 : 0.0)) : 2.0 * u; };
    double s = 0.0;
    for (int e = threadIdx.x; e < M_r; e += TR_BLK) {
        const int i = i0 + e;
        const double a = 1.0 - (double)A[i];
        s += pen(a);
        gA[i] += (float)(-c * dpen(a));
        if (h) {
            s += pen((double)h[i]);
            gh[i] += (float)(c * dpen((double)h[i]));
        }
    }
    for (int e = threadIdx.x; e < M_r * Lw; e += TR_BLK) {
        const int i = i0 + e / Lw, j = e % Lw;
        const double w = W[(size_t)i * Lw + j];
        s += gamma_w / Lw * pen(w);
        gW[(size_t)i * Lw + j] += (float)(c * gamma_w / Lw * dpen(w));
        if (shallow) {
            const double v = V[(size_t)j * M + i];
            s += gamma_v / Lw * pen(v);
            gV[(size_t)j * M + i] += (float)(c * gamma_v / Lw * dpen(v));
        }
    }
    const double t = block_sum(s, red);
    if (threadIdx.x == 0) mar[0] = c * t;
}

// loss = sum of the partials / (B N (T - T_w)) + MAR
__global__ void k_loss_final(const double *__restrict__ part, int np, double scale, const double *__restrict__ mar,
                             float *__restrict__ loss) {
    __shared__ double red[TR_BLK / 64];
    double s = 0.0;
    for (int e = threadIdx.x; e < np; e += blockDim.x) s += part[e];
    const double t = block_sum(s, red);
    if (threadIdx.x == 0) loss[0] = (float)(t * scale + (mar ? mar[0] : 0.0));
}

// one Adam step over the parameter segments (null segments are skipped)
struct ParamSeg {
    float *p[5];
    long n[5];
};

__global__ __launch_bounds__(TR_BLK) void k_adam(ParamSeg ps, const float *__restrict__ g, float *__restrict__ m,
                                                 float *__restrict__ v, long total, float lr, float b1, float b2,
                                                 float eps, float bc1, float bc2) {
    for (long e = blockIdx.x * (long)TR_BLK + threadIdx.x; e < total; e += (long)gridDim.x * TR_BLK) {
        long off = e;
        int k = 0;
        while (k < 5 && off >= ps.n[k]) {
            off -= ps.n[k];
            ++k;
        }
        if (k == 5 || !ps.p[k]) continue;
        const float ge = g[e];
        const float mn = b1 * m[e] + (1.f - b1) * ge;
        const float vn = b2 * v[e] + (1.f - b2) * ge * ge;
        m[e] = mn;
        v[e] = vn;
        ps.p[k][off] -= lr * (mn / bc1) / (sqrtf(vn / bc2) + eps);
    }
}

size_t train_partials() { return TR_NB; }

int launch_mse_loss_partial(const float *z, const float *x, int B, int T, int M, int N, int T_w, double *part,
                            hipStream_t st) {
    KTimer kt("k_mse_partial", st);
    hipLaunchKernelGGL(k_mse_partial, dim3(TR_NB), dim3(TR_BLK), 0, st, z, x, B, T, M, N, T_w, part);
    DEER_LAUNCH_CHECK("k_mse_partial");
    return DEER_OK;
}

int launch_mar(bool shallow, const float *A, const float *W, const float *V, const float *h, int M, int L, int M_r,
               float lam, int p, float gw, float gv, float *g, double *mar, hipStream_t st) {
    KTimer kt("k_mar", st);
    hipLaunchKernelGGL(k_mar, dim3(1), dim3(TR_BLK), 0, st, shallow ? 1 : 0, A, W, V, h, M, L, M_r, lam, p, gw, gv, g,
                       mar);
    DEER_LAUNCH_CHECK("k_mar");
    return DEER_OK;
}

int launch_loss_final(const double *part, double scale, const double *mar, float *loss, hipStream_t st) {
    hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(TR_BLK), 0, st, part, TR_NB, scale, mar, loss);
    DEER_LAUNCH_CHECK("k_loss_final");
    return DEER_OK;
}

int launch_adam(float *const *params, const long *sizes, const float *g, float *m, float *v, float lr, float b1,
                float b2, float eps, int step, hipStream_t st) {
    ParamSeg ps{};
    long total = 0;
    for (int k = 0; k < 5; ++k) {
        ps.p[k] = params[k];
        ps.n[k] = sizes[k];
        total += sizes[k];
    }
    const float bc1 = 1.f - powf(b1, (float)step), bc2 = 1.f - powf(b2, (float)step);
    const long want = (total + TR_BLK - 1) / TR_BLK;
    KTimer kt("k_adam", st);
    hipLaunchKernelGGL(k_adam, dim3((unsigned)(want < 1024 ? want : 1024)), dim3(TR_BLK), 0, st, ps, g, m, v, total, lr,
                       b1, b2, eps, bc1, bc2);
    DEER_LAUNCH_CHECK("k_adam");
    return DEER_OK;
}

}  // namespace deer
