// Sequential GTF baseline: the forward rollout z_s = F(z~_s) step by step and back-propagation
// through time, also step by step (the training the parallel solver replaces; the comparison
// of Fig. 1A).  One workgroup of 256 threads per sequence, weights in LDS, the steps in order:
// the batch is the only parallel dimension, as in a sequential scan vectorised over sequences.
//
// Model (both PLRNN kinds; the vanilla one is the shallow form with u = z~, L = M):
//   z~_s = z0 (or [x_0; 0]) at s = 0, else fl(fl(p z_{s-1}) + fl(alpha x_s)) on the forced
//   latents (eq. GTF; the same float32 operations as the parallel kernels);
//   u_s = h2 + W2 z~_s summed left to right with a rounding after every product and sum;
//   a_s = relu(u_s);  z_s = A z~_s + W1 a_s + h1.
// Adjoint (gradients appendix): lam_{T-1} = g_{T-1}, lam_s = g_s + P_alpha J_F(z~_{s+1})^T
// lam_{s+1} with J_F = diag(A) + W1 diag(m) W2, m = [u > 0]; gradients sum_s lam_s^T dF/dtheta:
//   dA += lam_s z~_s, dh1 += lam_s, dW1 += lam_s a_s^T, dW2 += q_s z~_s^T, dh2 += q_s with
//   q_s = m_s (W1^T lam_s).
#include "common.h"
#include "launch.h"

namespace deer {

namespace {

constexpr int kSeqThreads = 256;
constexpr int kSeqAcc = 32;   // gradient entries per thread and matrix: M L <= 256 * 32

__device__ __forceinline__ float pforce(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

// weights into LDS: W1 [M][L+1], W2 [L][M+1] (padded rows), A, h1 [M], h2 [L]
struct SeqLds {
    float *W1, *W2, *A, *h1, *h2, *zt, *a, *lam, *q;
};
__device__ __forceinline__ SeqLds seq_lds(float *sm, int M, int L, bool sh) {
    SeqLds s;
    s.W1 = sm;
    s.W2 = s.W1 + (size_t)M * (L + 1);
    s.A = s.W2 + (sh ? (size_t)L * (M + 1) : 0);
    s.h1 = s.A + M;
    s.h2 = s.h1 + M;
    s.zt = s.h2 + L;
    s.a = s.zt + M;
    s.lam = s.a + L;
    s.q = s.lam + M;
    return s;
}
__device__ __forceinline__ void seq_load_weights(const SeqLds &s, const float *A, const float *W1, const float *W2,
                                                 const float *h1, const float *h2, int M, int L, bool sh) {
    for (int e = threadIdx.x; e < M * L; e += blockDim.x) s.W1[(e / L) * (L + 1) + e % L] = W1[e];
    if (sh)
        for (int e = threadIdx.x; e < L * M; e += blockDim.x) s.W2[(e / M) * (M + 1) + e % M] = W2[e];
    for (int i = threadIdx.x; i < M; i += blockDim.x) {
        s.A[i] = A[i];
        s.h1[i] = h1 ? h1[i] : 0.f;
    }
    if (sh)
        for (int l = threadIdx.x; l < L; l += blockDim.x) s.h2[l] = h2 ? h2[l] : 0.f;
}

// u_l = h2_l + sum_j W2[l][j] z~_j (left to right, rounded after every operation)
__device__ __forceinline__ float seq_pre(const SeqLds &s, int l, int M) {
    float u = s.h2[l];
    const float *w = s.W2 + (size_t)l * (M + 1);
    for (int j = 0; j < M; ++j) u = __fadd_rn(u, __fmul_rn(w[j], s.zt[j]));
    return u;
}

}  // namespace

// Forward rollout.  act (shallow, may be null) receives a_s = relu(u_s) [B][T][L] for the
// backward pass.
template <bool SH>
__global__ __launch_bounds__(kSeqThreads) void k_seq_forward(const float *__restrict__ A, const float *__restrict__ W1,
                                                             const float *__restrict__ W2, const float *__restrict__ h1,
                                                             const float *__restrict__ h2, float alpha, int N,
                                                             const float *__restrict__ x, const float *__restrict__ z0,
                                                             float *__restrict__ z, float *__restrict__ act, int T,
                                                             int M, int L) {
    extern __shared__ float sm[];
    const SeqLds s = seq_lds(sm, M, L, SH);
    seq_load_weights(s, A, W1, W2, h1, h2, M, L, SH);
    const int b = blockIdx.x, tid = threadIdx.x;
    const float *xb = x + (size_t)b * (T + 1) * N;
    float *zb = z + (size_t)b * T * M;
    float zprev = 0.f;   // z_{s-1} of latent tid (the initial state at s = 0)
    if (tid < M) zprev = z0 ? z0[(size_t)b * M + tid] : (tid < N ? xb[tid] : 0.f);
    const float pi = pforce(tid, N, alpha);
    __syncthreads();
    for (int s0 = 0; s0 < T; ++s0) {
        float zt = 0.f;
        if (tid < M) {
            zt = (s0 == 0 || tid >= N) ? zprev : __fadd_rn(__fmul_rn(pi, zprev), __fmul_rn(alpha, xb[(size_t)s0 * N + tid]));
            s.zt[tid] = zt;
        }
        __syncthreads();
        if (SH) {
            for (int l = tid; l < L; l += kSeqThreads) {
                const float u = seq_pre(s, l, M);
                const float av = u > 0.f ? u : 0.f;
                s.a[l] = av;
                if (act) act[((size_t)b * T + s0) * L + l] = av;
            }
        } else if (tid < M) {
            s.a[tid] = zt > 0.f ? zt : 0.f;
        }
        __syncthreads();
        if (tid < M) {
            const float *w = s.W1 + (size_t)tid * (L + 1);
            float acc = 0.f;
            for (int k = 0; k < L; ++k) acc = fmaf(w[k], s.a[k], acc);
            const float F = fmaf(s.A[tid], zt, acc) + s.h1[tid];
            zb[(size_t)s0 * M + tid] = F;
            zprev = F;
        }
        // the next step writes zt only: every thread has passed the barrier after this
        // step's a, and a is written again only after the next barrier
    }
}

// Back-propagation through time for one sequence.  g null: the MSE seed scale * [z_s[:N] -
// x_{s+1}; 0].  lam (may be null) receives lam_s.  part receives the sequence's gradient sums
// [A M | W1 M L | h1 M | W2 L M | h2 L] (shallow) or [A M | W M M | h M] (vanilla).
template <bool SH>
__global__ __launch_bounds__(kSeqThreads) void k_seq_backward(
    const float *__restrict__ A, const float *__restrict__ W1, const float *__restrict__ W2,
    const float *__restrict__ h1, const float *__restrict__ h2, float alpha, int N, const float *__restrict__ x,
    const float *__restrict__ z0, const float *__restrict__ z, const float *__restrict__ act,
    const float *__restrict__ g, float seed_scale, float *__restrict__ lam, float *__restrict__ part, int T, int M,
    int L) {
    extern __shared__ float sm[];
    const SeqLds s = seq_lds(sm, M, L, SH);
    seq_load_weights(s, A, W1, W2, h1, h2, M, L, SH);
    const int b = blockIdx.x, tid = threadIdx.x;
    const float *xb = x + (size_t)b * (T + 1) * N;
    const float *zb = z + (size_t)b * T * M;
    const float pi = pforce(tid, N, alpha);
    const int ML = M * L;
    // this thread's entries of the two outer-product sums: e = tid + 256 q of W1 (row-major M x L,
    // packed i << 16 | k) and of W2 (row-major L x M)
    uint32_t e1[kSeqAcc], e2[kSeqAcc];
    float g1[kSeqAcc], g2[kSeqAcc];
#pragma unroll
    for (int q = 0; q < kSeqAcc; ++q) {
        const int e = tid + kSeqThreads * q;
        e1[q] = e < ML ? ((uint32_t)(e / L) << 16) | (uint32_t)(e % L) : 0xffffffffu;
        e2[q] = (SH && e < ML) ? ((uint32_t)(e / M) << 16) | (uint32_t)(e % M) : 0xffffffffu;
        g1[q] = 0.f;
        g2[q] = 0.f;
    }
    float gA = 0.f, gh1 = 0.f, gh2 = 0.f;
    // z~_s of latent tid
    auto forced = [&](int s0) {
        if (tid >= M) return 0.f;
        if (s0 == 0) return z0 ? z0[(size_t)b * M + tid] : (tid < N ? xb[tid] : 0.f);
        const float zp = zb[(size_t)(s0 - 1) * M + tid];
        return tid >= N ? zp : __fadd_rn(__fmul_rn(pi, zp), __fmul_rn(alpha, xb[(size_t)s0 * N + tid]));
    };
    // q = m (W1^T lam) for the lam and a in LDS, into s.q (L entries); the W2 and h2 sums of the
    // step whose z~ is in s.zt
    auto backprop_hidden = [&]() {
        for (int k = tid; k < L; k += kSeqThreads) {
            float v = 0.f;
            for (int i = 0; i < M; ++i) v = fmaf(s.W1[(size_t)i * (L + 1) + k], s.lam[i], v);
            s.q[k] = s.a[k] > 0.f ? v : 0.f;
        }
        __syncthreads();
        if (SH) {
            for (int l = tid; l < L; l += kSeqThreads) gh2 += s.q[l];
#pragma unroll
            for (int qq = 0; qq < kSeqAcc; ++qq)
                if (e2[qq] != 0xffffffffu) g2[qq] = fmaf(s.q[e2[qq] >> 16], s.zt[e2[qq] & 0xffffu], g2[qq]);
        }
    };
    for (int s0 = T - 1; s0 >= 0; --s0) {
        // lam_s = g_s + P (A lam_{s+1} + J^T part), with s.q = m_{s+1} (W1^T lam_{s+1})
        if (s0 < T - 1) backprop_hidden();
        float ls = 0.f, zt = 0.f;
        if (tid < M) {
            const float zs = zb[(size_t)s0 * M + tid];
            float gs;
            if (g) gs = g[((size_t)b * T + s0) * M + tid];
            else gs = tid < N ? seed_scale * (zs - xb[(size_t)(s0 + 1) * N + tid]) : 0.f;
            ls = gs;
            if (s0 < T - 1) {
                float w;
                if (SH) {
                    w = 0.f;
                    for (int k = 0; k < L; ++k) w = fmaf(s.W2[(size_t)k * (M + 1) + tid], s.q[k], w);
                } else {
                    w = s.q[tid];
                }
                ls = fmaf(pi, fmaf(s.A[tid], s.lam[tid], w), gs);
            }
            zt = forced(s0);
        }
        __syncthreads();   // every read of lam_{s+1}, q and the previous z~, a is done
        if (tid < M) {
            s.lam[tid] = ls;
            s.zt[tid] = zt;
            if (lam) lam[((size_t)b * T + s0) * M + tid] = ls;
            gA = fmaf(ls, zt, gA);
            gh1 += ls;
            if (!SH) s.a[tid] = zt > 0.f ? zt : 0.f;
        }
        if (SH)
            for (int l = tid; l < L; l += kSeqThreads) s.a[l] = act[((size_t)b * T + s0) * L + l];
        __syncthreads();
        // dW1 += lam_s a_s^T
#pragma unroll
        for (int qq = 0; qq < kSeqAcc; ++qq)
            if (e1[qq] != 0xffffffffu) g1[qq] = fmaf(s.lam[e1[qq] >> 16], s.a[e1[qq] & 0xffffu], g1[qq]);
        __syncthreads();
    }
    backprop_hidden();   // the W2 and h2 sums of step 0
    // this sequence's sums
    float *pA = part + (size_t)b * (SH ? (size_t)2 * M + 2 * (size_t)ML + L : (size_t)2 * M + ML);
    float *pW1 = pA + M, *ph1 = pW1 + ML, *pW2 = ph1 + M, *ph2 = pW2 + ML;
    if (tid < M) {
        pA[tid] = gA;
        ph1[tid] = gh1;
    }
#pragma unroll
    for (int qq = 0; qq < kSeqAcc; ++qq) {
        const int e = tid + kSeqThreads * qq;
        if (e < ML) pW1[e] = g1[qq];
        if (SH && e < ML) pW2[e] = g2[qq];
    }
    if (SH)
        for (int l = tid; l < L; l += kSeqThreads) ph2[l] = gh2;
}

// sum over the B sequences' parts (float64), into the gradient outputs
__global__ void k_seq_grads_sum(const float *__restrict__ part, int B, int M, int L, int SH, deer_grads gr) {
    const int ML = M * L;
    const size_t per = SH ? (size_t)2 * M + 2 * (size_t)ML + L : (size_t)2 * M + ML;
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < per; e += (size_t)gridDim.x * blockDim.x) {
        double acc = 0.0;
        for (int b = 0; b < B; ++b) acc += (double)part[(size_t)b * per + e];
        const float v = (float)acc;
        size_t o = e;
        if (o < (size_t)M) { if (gr.A) gr.A[o] = v; continue; }
        o -= M;
        if (o < (size_t)ML) { if (gr.W) gr.W[o] = v; continue; }
        o -= ML;
        if (o < (size_t)M) { if (gr.h) gr.h[o] = v; continue; }
        o -= M;
        if (o < (size_t)ML) { if (gr.W2) gr.W2[o] = v; continue; }
        o -= ML;
        if (gr.h2) gr.h2[o] = v;
    }
}

size_t seq_lds_bytes(int M, int L, bool sh) {
    return sizeof(float) * ((size_t)M * (L + 1) + (sh ? (size_t)L * (M + 1) : 0) + 3 * (size_t)M + 3 * (size_t)L + M);
}

size_t seq_part_floats(int M, int L, bool sh) {
    return sh ? (size_t)2 * M + 2 * (size_t)M * L + L : (size_t)2 * M + (size_t)M * L;
}

int seq_check(int M, int L, bool sh) {
    if (M > kSeqThreads || (sh && L > kSeqThreads) || (size_t)M * L > (size_t)kSeqThreads * kSeqAcc ||
        seq_lds_bytes(M, L, sh) > 160 * 1024)
        return -1;
    return 0;
}

int launch_seq_forward(const SeqArgs &a, float *z, float *act, hipStream_t st) {
    const size_t lds = seq_lds_bytes(a.M, a.L, a.sh);
    KTimer kt("k_seq_forward", st);
    if (a.sh) {
        DEER_HIP(hipFuncSetAttribute((const void *)k_seq_forward<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds));
        hipLaunchKernelGGL(k_seq_forward<true>, dim3(a.B), dim3(kSeqThreads), lds, st, a.A, a.W1, a.W2, a.h1, a.h2,
                           a.alpha, a.N, a.x, a.z0, z, act, a.T, a.M, a.L);
    } else {
        DEER_HIP(hipFuncSetAttribute((const void *)k_seq_forward<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds));
        hipLaunchKernelGGL(k_seq_forward<false>, dim3(a.B), dim3(kSeqThreads), lds, st, a.A, a.W1, a.W2, a.h1, a.h2,
                           a.alpha, a.N, a.x, a.z0, z, act, a.T, a.M, a.L);
    }
    DEER_LAUNCH_CHECK("k_seq_forward");
    return DEER_OK;
}

int launch_seq_backward(const SeqArgs &a, const float *z, const float *act, const float *g, float seed_scale,
                        float *lam, float *part, const deer_grads *gr, hipStream_t st) {
    const size_t lds = seq_lds_bytes(a.M, a.L, a.sh);
    {
        KTimer kt("k_seq_backward", st);
        if (a.sh) {
            DEER_HIP(hipFuncSetAttribute((const void *)k_seq_backward<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds));
            hipLaunchKernelGGL(k_seq_backward<true>, dim3(a.B), dim3(kSeqThreads), lds, st, a.A, a.W1, a.W2, a.h1,
                               a.h2, a.alpha, a.N, a.x, a.z0, z, act, g, seed_scale, lam, part, a.T, a.M, a.L);
        } else {
            DEER_HIP(hipFuncSetAttribute((const void *)k_seq_backward<false>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
            hipLaunchKernelGGL(k_seq_backward<false>, dim3(a.B), dim3(kSeqThreads), lds, st, a.A, a.W1, a.W2, a.h1,
                               a.h2, a.alpha, a.N, a.x, a.z0, z, act, g, seed_scale, lam, part, a.T, a.M, a.L);
        }
        DEER_LAUNCH_CHECK("k_seq_backward");
    }
    if (gr) {
        KTimer kt("k_seq_grads_sum", st);
        const size_t per = seq_part_floats(a.M, a.L, a.sh);
        const unsigned grid = (unsigned)((per + 255) / 256);
        hipLaunchKernelGGL(k_seq_grads_sum, dim3(grid), dim3(256), 0, st, (const float *)part, a.B, a.M, a.L,
                           a.sh ? 1 : 0, *gr);
        DEER_LAUNCH_CHECK("k_seq_grads_sum");
    }
    return DEER_OK;
}

}  // namespace deer
