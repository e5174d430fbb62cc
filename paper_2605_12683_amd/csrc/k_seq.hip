// Sequential GTF baseline: the forward rollout z_s = F(z~_s) step by step and back-propagation
// through time, also step by step (the training the parallel solver replaces; the comparison
// of Fig. 1A).  One wave per sequence, the batch being the only parallel dimension, as in a
// sequential scan vectorised over sequences.  A wave needs no workgroup barrier: its lanes
// exchange data through LDS, synchronised within the wave.  Weights live in LDS; the per-step
// inputs (x, and for the backward pass z, g and the hidden activations) are staged into LDS a
// chunk of steps at a time, so the loop does not wait for memory at every step; the outer-
// product gradient sums are formed per chunk from buffered (lambda, a) and (q, z~) rows.
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

constexpr int kW = 64;                  // one wave per sequence
constexpr int kSeqMaxDim = 256;         // M, L <= 256: at most four outputs per lane
constexpr int kNQ = kSeqMaxDim / kW;
constexpr size_t kSeqLdsFloats = 38 * 1024;   // LDS budget of a sequence (152 KiB)

__device__ __forceinline__ float pforce(int i, int N, float alpha) { return i < N ? __fsub_rn(1.0f, alpha) : 1.0f; }

// sum_k w[k * stride] v[k], k < n, in four interleaved partial sums (short dependency chains)
__device__ __forceinline__ float seq_dot(const float *w, int stride, const float *v, int n) {
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    int k = 0;
    for (; k + 4 <= n; k += 4) {
        a0 = fmaf(w[(size_t)k * stride], v[k], a0);
        a1 = fmaf(w[(size_t)(k + 1) * stride], v[k + 1], a1);
        a2 = fmaf(w[(size_t)(k + 2) * stride], v[k + 2], a2);
        a3 = fmaf(w[(size_t)(k + 3) * stride], v[k + 3], a3);
    }
    for (; k < n; ++k) a0 = fmaf(w[(size_t)k * stride], v[k], a0);
    return (a0 + a1) + (a2 + a3);
}

// LDS: W1 [M][L+1], W2 [L][M+1], A, h1 [M], h2 [L], zt [M], a [L], lam [M], q [L], then the
// chunk buffers
struct SeqLds {
    float *W1, *W2, *A, *h1, *h2, *zt, *a, *lam, *q, *buf;
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
    s.buf = s.q + L;
    return s;
}
__host__ __device__ inline size_t seq_fixed_floats(int M, int L, bool sh) {
    return (size_t)M * (L + 1) + (sh ? (size_t)L * (M + 1) : 0) + 4 * (size_t)M + 4 * (size_t)L;
}
// floats a chunk step needs: forward x rows; backward z, x, g and a rows and the lam, z~, a, q
// rows of the gradient sums (plus one more z and x row per chunk)
__host__ __device__ inline size_t seq_step_floats(int M, int L, int N, bool sh, bool has_g, bool backward) {
    return backward ? (size_t)M + N + (has_g ? M : 0) + (sh ? L : 0) + 2 * (size_t)(M + L) : (size_t)(N > 0 ? N : 1);
}
__host__ __device__ inline int seq_chunk(int M, int L, int N, bool sh, bool has_g, bool backward) {
    const size_t fixed = seq_fixed_floats(M, L, sh) + (backward ? (size_t)M + N : 0);
    if (fixed + 64 > kSeqLdsFloats) return 0;
    size_t ch = (kSeqLdsFloats - fixed) / seq_step_floats(M, L, N, sh, has_g, backward);
    if (ch > 256) ch = 256;
    return (int)ch;
}

__device__ __forceinline__ void seq_load_weights(const SeqLds &s, const float *A, const float *W1, const float *W2,
                                                 const float *h1, const float *h2, int M, int L, bool sh, int lane) {
    for (int e = lane; e < M * L; e += kW) s.W1[(e / L) * (L + 1) + e % L] = W1[e];
    if (sh)
        for (int e = lane; e < L * M; e += kW) s.W2[(e / M) * (M + 1) + e % M] = W2[e];
    for (int i = lane; i < M; i += kW) {
        s.A[i] = A[i];
        s.h1[i] = h1 ? h1[i] : 0.f;
    }
    for (int l = lane; l < L; l += kW) s.h2[l] = (sh && h2) ? h2[l] : 0.f;
}

// rows [r0, r0 + n) of a row-major array of width w into LDS, lanes striding
__device__ __forceinline__ void seq_stage(float *dst, const float *src, size_t r0, int n, int w, int lane) {
    const size_t cnt = (size_t)n * w;
    const float *p = src + r0 * w;
    for (size_t e = lane; e < cnt; e += kW) dst[e] = p[e];
}

}  // namespace

// Forward rollout.  act (shallow, may be null) receives a_s = relu(u_s) [B][T][L] for the
// backward pass.
template <bool SH>
__global__ __launch_bounds__(kW) void k_seq_forward(const float *__restrict__ A, const float *__restrict__ W1,
                                                    const float *__restrict__ W2, const float *__restrict__ h1,
                                                    const float *__restrict__ h2, float alpha, int N,
                                                    const float *__restrict__ x, const float *__restrict__ z0,
                                                    float *__restrict__ z, float *__restrict__ act, int T, int M,
                                                    int L, int CH) {
    extern __shared__ float sm[];
    const int lane = threadIdx.x, b = blockIdx.x;
    const SeqLds s = seq_lds(sm, M, L, SH);
    seq_load_weights(s, A, W1, W2, h1, h2, M, L, SH, lane);
    const float *xb = x + (size_t)b * (T + 1) * N;
    float *zb = z + (size_t)b * T * M;
    float *xs = s.buf;   // x rows of the chunk [CH][N]
    float zprev[kNQ];    // z_{s-1} of latents lane + 64 r
#pragma unroll
    for (int r = 0; r < kNQ; ++r) {
        const int i = lane + kW * r;
        zprev[r] = i < M ? (z0 ? z0[(size_t)b * M + i] : (i < N ? xb[i] : 0.f)) : 0.f;
    }
    for (int c0 = 0; c0 < T; c0 += CH) {
        const int n = min(CH, T - c0);
        wave_lds_sync();
        if (N > 0) seq_stage(xs, xb, c0, n, N, lane);
        wave_lds_sync();
        for (int t = 0; t < n; ++t) {
            const int s0 = c0 + t;
            float zt[kNQ];
#pragma unroll
            for (int r = 0; r < kNQ; ++r) {
                const int i = lane + kW * r;
                zt[r] = 0.f;
                if (i < M) {
                    zt[r] = (s0 == 0 || i >= N) ? zprev[r]
                                                : __fadd_rn(__fmul_rn(pforce(i, N, alpha), zprev[r]),
                                                            __fmul_rn(alpha, xs[(size_t)t * N + i]));
                    s.zt[i] = zt[r];
                }
            }
            wave_lds_sync();
            if (SH) {
                for (int l = lane; l < L; l += kW) {
                    float u = s.h2[l];
                    const float *w = s.W2 + (size_t)l * (M + 1);
                    for (int j = 0; j < M; ++j) u = __fadd_rn(u, __fmul_rn(w[j], s.zt[j]));
                    const float av = u > 0.f ? u : 0.f;
                    s.a[l] = av;
                    if (act) act[((size_t)b * T + s0) * L + l] = av;
                }
            } else {
#pragma unroll
                for (int r = 0; r < kNQ; ++r) {
                    const int i = lane + kW * r;
                    if (i < M) s.a[i] = zt[r] > 0.f ? zt[r] : 0.f;
                }
            }
            wave_lds_sync();
#pragma unroll
            for (int r = 0; r < kNQ; ++r) {
                const int i = lane + kW * r;
                if (i < M) {
                    const float F = fmaf(s.A[i], zt[r], seq_dot(s.W1 + (size_t)i * (L + 1), 1, s.a, L)) + s.h1[i];
                    zb[(size_t)s0 * M + i] = F;
                    zprev[r] = F;
                }
            }
        }
    }
}

// Back-propagation through time for one sequence.  g null: the MSE seed scale * [z_s[:N] -
// x_{s+1}; 0].  lam (may be null) receives lam_s.  part receives the sequence's gradient sums
// [A M | W1 M L | h1 M | W2 L M | h2 L] (shallow) or [A M | W M M | h M] (vanilla).
template <bool SH>
__global__ __launch_bounds__(kW) void k_seq_backward(
    const float *__restrict__ A, const float *__restrict__ W1, const float *__restrict__ W2,
    const float *__restrict__ h1, const float *__restrict__ h2, float alpha, int N, const float *__restrict__ x,
    const float *__restrict__ z0, const float *__restrict__ z, const float *__restrict__ act,
    const float *__restrict__ g, float seed_scale, float *__restrict__ lam, float *__restrict__ part, int T, int M,
    int L, int CH) {
    extern __shared__ float sm[];
    const int lane = threadIdx.x, b = blockIdx.x;
    const SeqLds s = seq_lds(sm, M, L, SH);
    seq_load_weights(s, A, W1, W2, h1, h2, M, L, SH, lane);
    const float *xb = x + (size_t)b * (T + 1) * N;
    const float *zb = z + (size_t)b * T * M;
    const int ML = M * L;
    float *pA = part + (size_t)b * (SH ? (size_t)2 * M + 2 * (size_t)ML + L : (size_t)2 * M + ML);
    float *pW1 = pA + M, *ph1 = pW1 + ML, *pW2 = ph1 + M, *ph2 = pW2 + ML;
    for (int e = lane; e < ML; e += kW) {
        pW1[e] = 0.f;
        if (SH) pW2[e] = 0.f;
    }
    // chunk buffers: z rows c0-1 .. c1-1, x rows c0 .. c1, g and a rows c0 .. c1-1, then the
    // rows of the gradient sums (lam, z~, a, q per step of the chunk)
    float *zs = s.buf;                              // [CH + 1][M], row 0 = z_{c0-1}
    float *xs = zs + (size_t)(CH + 1) * M;          // [CH + 1][N], row 0 = x_{c0}
    float *gs = xs + (size_t)(CH + 1) * N;          // [CH][M] if g
    float *as = gs + (g ? (size_t)CH * M : 0);      // [CH][L] shallow
    float *rl = as + (SH ? (size_t)CH * L : 0);     // lam rows [CH][M]
    float *rz = rl + (size_t)CH * M;                // z~ rows [CH][M]
    float *ra = rz + (size_t)CH * M;                // a rows [CH][L]
    float *rq = ra + (size_t)CH * L;                // q rows [CH][L]
    float gA[kNQ], gh1[kNQ], gh2[kNQ];
#pragma unroll
    for (int r = 0; r < kNQ; ++r) gA[r] = gh1[r] = gh2[r] = 0.f;
    bool first = true;   // s = T - 1: lam = g
    for (int c1 = T; c1 > 0; c1 -= CH) {
        const int c0 = max(0, c1 - CH), n = c1 - c0;
        wave_lds_sync();
        if (c0 > 0) seq_stage(zs, zb, c0 - 1, n + 1, M, lane);
        else seq_stage(zs + M, zb, 0, n, M, lane);
        if (N > 0) seq_stage(xs, xb, c0, n + 1, N, lane);
        if (g) seq_stage(gs, g + (size_t)b * T * M, c0, n, M, lane);
        if (SH) seq_stage(as, act + (size_t)b * T * L, c0, n, L, lane);
        wave_lds_sync();
        for (int t = n - 1; t >= 0; --t) {
            const int s0 = c0 + t;
            // lam_s = g_s + P (A lam_{s+1} + W2^T q_{s+1}), z~_s, a_s
            float ls[kNQ], zt[kNQ];
#pragma unroll
            for (int r = 0; r < kNQ; ++r) {
                const int i = lane + kW * r;
                ls[r] = zt[r] = 0.f;
                if (i >= M) continue;
                const float gv = g ? gs[(size_t)t * M + i]
                                   : (i < N ? seed_scale * (zs[(size_t)(t + 1) * M + i] - xs[(size_t)(t + 1) * N + i])
                                            : 0.f);
                ls[r] = gv;
                if (!first) {
                    const float w = SH ? seq_dot(s.W2 + i, M + 1, s.q, L) : s.q[i];
                    ls[r] = fmaf(pforce(i, N, alpha), fmaf(s.A[i], s.lam[i], w), gv);
                }
                if (s0 == 0) {
                    zt[r] = z0 ? z0[(size_t)b * M + i] : (i < N ? xb[i] : 0.f);
                } else {
                    const float zp = zs[(size_t)t * M + i];
                    zt[r] = i >= N ? zp
                                   : __fadd_rn(__fmul_rn(pforce(i, N, alpha), zp), __fmul_rn(alpha, xs[(size_t)t * N + i]));
                }
            }
            first = false;
            wave_lds_sync();   // every read of lam_{s+1} and q_{s+1} is done
#pragma unroll
            for (int r = 0; r < kNQ; ++r) {
                const int i = lane + kW * r;
                if (i >= M) continue;
                s.lam[i] = ls[r];
                s.zt[i] = zt[r];
                rl[(size_t)t * M + i] = ls[r];
                rz[(size_t)t * M + i] = zt[r];
                if (lam) lam[((size_t)b * T + s0) * M + i] = ls[r];
                gA[r] = fmaf(ls[r], zt[r], gA[r]);
                gh1[r] += ls[r];
                if (!SH) {
                    const float av = zt[r] > 0.f ? zt[r] : 0.f;
                    s.a[i] = av;
                    ra[(size_t)t * L + i] = av;
                }
            }
            if (SH)
                for (int l = lane; l < L; l += kW) {
                    const float av = as[(size_t)t * L + l];
                    s.a[l] = av;
                    ra[(size_t)t * L + l] = av;
                }
            wave_lds_sync();
            // q_s = m_s (W1^T lam_s): the next step's W2^T q and this step's W2, h2 sums
#pragma unroll
            for (int r = 0; r < kNQ; ++r) {
                const int k = lane + kW * r;
                if (k >= L) continue;
                const float v = seq_dot(s.W1 + k, L + 1, s.lam, M);
                const float qv = s.a[k] > 0.f ? v : 0.f;
                s.q[k] = qv;
                rq[(size_t)t * L + k] = qv;
                gh2[r] += qv;
            }
            wave_lds_sync();
        }
        // the chunk's outer-product sums: W1 += sum_t lam_t a_t^T, W2 += sum_t q_t z~_t^T
        for (int e = lane; e < ML; e += kW) {
            const int i = e / L, k = e - i * L;
            float acc = 0.f;
            for (int t = 0; t < n; ++t) acc = fmaf(rl[(size_t)t * M + i], ra[(size_t)t * L + k], acc);
            pW1[e] += acc;
            if (SH) {
                const int l = e / M, j = e - l * M;
                float acc2 = 0.f;
                for (int t = 0; t < n; ++t) acc2 = fmaf(rq[(size_t)t * L + l], rz[(size_t)t * M + j], acc2);
                pW2[e] += acc2;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kNQ; ++r) {
        const int i = lane + kW * r;
        if (i < M) {
            pA[i] = gA[r];
            ph1[i] = gh1[r];
        }
        if (SH && i < L) ph2[i] = gh2[r];
    }
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

size_t seq_part_floats(int M, int L, bool sh) {
    return sh ? (size_t)2 * M + 2 * (size_t)M * L + L : (size_t)2 * M + (size_t)M * L;
}

int seq_check(int M, int L, bool sh) {
    if (M > kSeqMaxDim || L > kSeqMaxDim || (size_t)M * L > 8192) return -1;
    // the largest stage: backward with a cotangent and the largest forcing count N = M
    if (seq_chunk(M, L, M, sh, true, true) < 8) return -1;
    return 0;
}

int launch_seq_forward(const SeqArgs &a, float *z, float *act, hipStream_t st) {
    const int CH = seq_chunk(a.M, a.L, a.N, a.sh, false, false);
    const size_t lds = sizeof(float) * (seq_fixed_floats(a.M, a.L, a.sh) +
                                        (size_t)CH * seq_step_floats(a.M, a.L, a.N, a.sh, false, false));
    KTimer kt("k_seq_forward", st);
#define SEQF(SHV)                                                                                                  \
    do {                                                                                                           \
        DEER_HIP(hipFuncSetAttribute((const void *)k_seq_forward<SHV>, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                     (int)lds));                                                                   \
        hipLaunchKernelGGL(k_seq_forward<SHV>, dim3(a.B), dim3(kW), lds, st, a.A, a.W1, a.W2, a.h1, a.h2, a.alpha, \
                           a.N, a.x, a.z0, z, act, a.T, a.M, a.L, CH);                                             \
    } while (0)
    if (a.sh) SEQF(true);
    else SEQF(false);
#undef SEQF
    DEER_LAUNCH_CHECK("k_seq_forward");
    return DEER_OK;
}

int launch_seq_backward(const SeqArgs &a, const float *z, const float *act, const float *g, float seed_scale,
                        float *lam, float *part, const deer_grads *gr, hipStream_t st) {
    const bool hg = g != nullptr;
    const int CH = seq_chunk(a.M, a.L, a.N, a.sh, hg, true);
    const size_t lds = sizeof(float) * (seq_fixed_floats(a.M, a.L, a.sh) + (size_t)a.M + a.N +
                                        (size_t)CH * seq_step_floats(a.M, a.L, a.N, a.sh, hg, true));
    {
        KTimer kt("k_seq_backward", st);
#define SEQB(SHV)                                                                                                   \
    do {                                                                                                            \
        DEER_HIP(hipFuncSetAttribute((const void *)k_seq_backward<SHV>, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                     (int)lds));                                                                    \
        hipLaunchKernelGGL(k_seq_backward<SHV>, dim3(a.B), dim3(kW), lds, st, a.A, a.W1, a.W2, a.h1, a.h2, a.alpha, \
                           a.N, a.x, a.z0, z, act, g, seed_scale, lam, part, a.T, a.M, a.L, CH);                    \
    } while (0)
        if (a.sh) SEQB(true);
        else SEQB(false);
#undef SEQB
        DEER_LAUNCH_CHECK("k_seq_backward");
    }
    if (gr) {
        KTimer kt("k_seq_grads_sum", st);
        const size_t pf = seq_part_floats(a.M, a.L, a.sh);
        const unsigned grid = (unsigned)((pf + 255) / 256);
        hipLaunchKernelGGL(k_seq_grads_sum, dim3(grid), dim3(256), 0, st, (const float *)part, a.B, a.M, a.L,
                           a.sh ? 1 : 0, *gr);
        DEER_LAUNCH_CHECK("k_seq_grads_sum");
    }
    return DEER_OK;
}

}  // namespace deer
