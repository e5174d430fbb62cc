// Diagonal complex linear recurrence (the LSSM's training-time scan, eq. shplrnn_ssm with a
// diagonal complex A; Alg. LSSM):
//   forward  y_t = lam * y_{t-1} + b_t,              y_0 = 0
//   reverse  y_{t-1} = conj(lam) * y_t + b_{t-1},    y_T = b_T   (the transpose, on C = R^2)
// Every channel is an independent first-order recurrence; the work is bandwidth bound.
//
// Three kernels per scan, all with the same tile: 16 channels (one 128-byte row segment per
// timestep) x CH = 1024 consecutive positions; a lane owns S = 32 consecutive positions of
// one channel in registers (lane = 16 j + ch, wave w: sub-chunk u = 4 w + j):
//   k_diag_chunk<REDUCE>  chunk aggregates A_q = local scan of the chunk from zero
//   k_diag_carry          X_q = sum_{q' < q} Lambda^(q-1-q') A_q' (Lambda = lam^CH), per channel
//   k_diag_chunk<FIXUP>   re-scan of the chunk from X_q, written out
// Positions are logical: reverse scans run over time T-1-p.  b may be given, or formed on
// the fly as b_t = Bc u_t with u_t = x_{t-1} (input projection fused, K inputs).
#include <stdlib.h>

#include "common.h"
#include "launch.h"

namespace deer {

typedef float v2f __attribute__((ext_vector_type(2)));

namespace {
constexpr int DTC = 16;                  // channels per tile
constexpr int DS = 16;                   // positions per lane
constexpr int DNW = 8;                   // waves per block
constexpr int DCH = DNW * 4 * DS;        // positions per chunk (1024)

struct cd {
    double re, im;
};
__device__ __forceinline__ cd cmul(cd a, cd b) { return {a.re * b.re - a.im * b.im, a.re * b.im + a.im * b.re}; }
__device__ __forceinline__ cd cpow(cd a, long e) {
    cd r = {1.0, 0.0};
    while (e > 0) {
        if (e & 1) r = cmul(r, a);
        a = cmul(a, a);
        e >>= 1;
    }
    return r;
}
}  // namespace

template <bool FIXUP>
__global__ __launch_bounds__(DNW * 64) void k_diag_chunk(const float *__restrict__ lam, int conj_lam,
                                                        const float *__restrict__ bin, const float *__restrict__ Bc,
                                                        int K, const float *__restrict__ u, int rev, int B, int T,
                                                        int M, int ntile, int nq, float *__restrict__ agg,
                                                        const float *__restrict__ carry, float *__restrict__ yout) {
    __shared__ float2 sub[DNW * 4][DTC];
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, j = lane >> 4, ch = lane & 15;
    const int usub = w * 4 + j;
    const int q = blockIdx.x % nq;
    const int st = blockIdx.x / nq;                 // (sequence, channel tile)
    const int b = st / ntile, tile = st % ntile;
    const int m = tile * DTC + ch;
    const bool mok = m < M;
    float lr = 0.f, li = 0.f;
    if (mok) {
        lr = lam[2 * m];
        li = conj_lam ? -lam[2 * m + 1] : lam[2 * m + 1];
    }
    // input projection row of this channel (fused path)
    float br[4] = {0.f, 0.f, 0.f, 0.f}, bi[4] = {0.f, 0.f, 0.f, 0.f};
    if (!bin && mok) {
        for (int k = 0; k < K && k < 4; ++k) {
            br[k] = Bc[(m * K + k) * 2];
            bi[k] = Bc[(m * K + k) * 2 + 1];
        }
    }
    const long p0 = (long)q * DCH + (long)usub * DS;   // first logical position of this lane
    float2 bv[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const long p = p0 + s;
        float2 v = make_float2(0.f, 0.f);
        if (mok && p < T) {
            const long tau = rev ? (T - 1 - p) : p;
            if (bin) {
                v = *reinterpret_cast<const float2 *>(bin + (((long)b * T + tau) * M + m) * 2);
            } else {
                const float *uu = u + ((long)b * (T + 1) + tau) * K;     // u_{tau+1} = x_tau
                for (int k = 0; k < K && k < 4; ++k) {
                    const float uk = uu[k];
                    v.x = fmaf(br[k], uk, v.x);
                    v.y = fmaf(bi[k], uk, v.y);
                }
            }
        }
        bv[s] = v;
    }
    // local scan of this lane's positions from zero
    float er = 0.f, ei = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const float nr = fmaf(lr, er, fmaf(-li, ei, bv[s].x));
        const float ni = fmaf(lr, ei, fmaf(li, er, bv[s].y));
        er = nr;
        ei = ni;
    }
    sub[usub][ch] = make_float2(er, ei);
    __syncthreads();
    // exclusive prefix over the sub-chunks before this one: P_u = sum_{u'<u} L^(u-1-u') e_u'
    const cd lamd = {(double)lr, (double)li};
    const cd Ls = cpow(lamd, DS);
    const float Lsr = (float)Ls.re, Lsi = (float)Ls.im;
    float pr = 0.f, pi = 0.f;
    for (int k = 0; k < usub; ++k) {
        const float2 e = sub[k][ch];
        const float nr = fmaf(Lsr, pr, fmaf(-Lsi, pi, e.x));
        const float ni = fmaf(Lsr, pi, fmaf(Lsi, pr, e.y));
        pr = nr;
        pi = ni;
    }
    if (!FIXUP) {
        if (usub == DNW * 4 - 1 && mok) {
            // chunk aggregate = L^S * P_last + e_last
            const float ar = fmaf(Lsr, pr, fmaf(-Lsi, pi, er));
            const float ai = fmaf(Lsr, pi, fmaf(Lsi, pr, ei));
            reinterpret_cast<float2 *>(agg)[((long)st * nq + q) * DTC + ch] = make_float2(ar, ai);
        }
        return;
    }
    // start state of this lane: lam^(u S) X_q + P_u
    float yr = pr, yi = pi;
    if (q > 0 && mok) {
        const float2 X = reinterpret_cast<const float2 *>(carry)[((long)st * nq + q) * DTC + ch];
        const cd Lu = cpow(lamd, (long)usub * DS);
        const double xr = Lu.re * X.x - Lu.im * X.y, xi = Lu.re * X.y + Lu.im * X.x;
        yr = (float)((double)pr + xr);
        yi = (float)((double)pi + xi);
    }
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const float nr = fmaf(lr, yr, fmaf(-li, yi, bv[s].x));
        const float ni = fmaf(lr, yi, fmaf(li, yr, bv[s].y));
        yr = nr;
        yi = ni;
        const long p = p0 + s;
        if (mok && p < T) {
            const long tau = rev ? (T - 1 - p) : p;
            *reinterpret_cast<float2 *>(yout + (((long)b * T + tau) * M + m) * 2) = make_float2(yr, yi);
        }
    }
}

// ---------------------------------------------------------------------------------------
// Single-pass variant (one HBM read of b, one write of y): chunks are processed in ticket
// order per chain (chain = (sequence, channel tile)); each block publishes its chunk
// aggregate, looks back over its predecessors' published values until it meets an inclusive
// prefix (decoupled look-back), publishes its own inclusive prefix and re-scans its chunk
// from the carry held in registers.  Every published 64-bit word is (valid << 32 | float
// bits), written and read with relaxed device-scope atomics, so a reader needs no ordering
// between words: it waits until every word it needs carries the valid flag.
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ void pub_word(unsigned long long *p, float v) {
    const unsigned long long w = (1ull << 32) | (unsigned long long)(uint32_t)__float_as_uint(v);
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <bool PROJ>
__global__ __launch_bounds__(DNW * 64) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_diag_scan_lb(const float *__restrict__ lam, int conj_lam,
                                                          const float *__restrict__ bin, const float *__restrict__ Bc,
                                                          int K, const float *__restrict__ u, int rev, int B, int T,
                                                          int M, int ntile, int nq, unsigned int *__restrict__ ticket,
                                                          unsigned long long *__restrict__ aggw,
                                                          unsigned long long *__restrict__ incw,
                                                          float *__restrict__ yout) {
    __shared__ float2 sub[DNW * 4][DTC];
    __shared__ float2 xq[DTC];
    __shared__ float xs[PROJ ? DCH * 4 : 1];
    __shared__ unsigned int vid_s;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, j = lane >> 4, ch = lane & 15;
    const int usub = w * 4 + j;
    if (tid == 0) vid_s = atomicAdd(ticket, 1u);
    __syncthreads();
    const unsigned int vid = vid_s;
    const int nchain = B * ntile;
    const int q = (int)(vid / nchain);
    const int st = (int)(vid % nchain);
    const int b = st / ntile, tile = st % ntile;
    const int m = tile * DTC + ch;
    const bool mok = m < M;
    float lr = 0.f, li = 0.f;
    if (mok) {
        lr = lam[2 * m];
        li = conj_lam ? -lam[2 * m + 1] : lam[2 * m + 1];
    }
    float br[4] = {0.f, 0.f, 0.f, 0.f}, bi[4] = {0.f, 0.f, 0.f, 0.f};
    if (PROJ && mok) {
        for (int k = 0; k < K && k < 4; ++k) {
            br[k] = Bc[(m * K + k) * 2];
            bi[k] = Bc[(m * K + k) * 2 + 1];
        }
    }
    const long p0 = (long)q * DCH + (long)usub * DS;
    if (PROJ) {
        // inputs of this chunk staged in LDS with coalesced loads (forward only: tau = p)
        const long n = (long)DCH * K;
        for (long e = tid; e < n; e += DNW * 64) {
            const long p = (long)q * DCH + e / K;
            xs[e] = p < T ? u[((long)b * (T + 1) + p) * K + (e % K)] : 0.f;
        }
        __syncthreads();
    }
    float2 bv[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const long p = p0 + s;
        float2 v = make_float2(0.f, 0.f);
        if (mok && p < T) {
            const long tau = rev ? (T - 1 - p) : p;
            if (!PROJ) {
                const v2f t2 = __builtin_nontemporal_load(reinterpret_cast<const v2f *>(bin + (((long)b * T + tau) * M + m) * 2));
                v = make_float2(t2.x, t2.y);
            } else {
                const float *uu = xs + (long)(usub * DS + s) * K;
                for (int k = 0; k < K && k < 4; ++k) {
                    const float uk = uu[k];
                    v.x = fmaf(br[k], uk, v.x);
                    v.y = fmaf(bi[k], uk, v.y);
                }
            }
        }
        bv[s] = v;
    }
    float er = 0.f, ei = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const float nr = fmaf(lr, er, fmaf(-li, ei, bv[s].x));
        const float ni = fmaf(lr, ei, fmaf(li, er, bv[s].y));
        er = nr;
        ei = ni;
    }
    sub[usub][ch] = make_float2(er, ei);
    __syncthreads();
    const cd lamd = {(double)lr, (double)li};
    const cd Ls = cpow(lamd, DS);
    const float Lsr = (float)Ls.re, Lsi = (float)Ls.im;
    float pr = 0.f, pi = 0.f;
    for (int k = 0; k < usub; ++k) {
        const float2 e = sub[k][ch];
        const float nr = fmaf(Lsr, pr, fmaf(-Lsi, pi, e.x));
        const float ni = fmaf(Lsr, pi, fmaf(Lsi, pr, e.y));
        pr = nr;
        pi = ni;
    }
    if (usub == DNW * 4 - 1) {
        // the lanes of the last sub-chunk own the chunk aggregate and do the look-back
        const float ar = fmaf(Lsr, pr, fmaf(-Lsi, pi, er));
        const float ai = fmaf(Lsr, pi, fmaf(Lsi, pr, ei));
        const size_t me = (((size_t)st * nq + q) * DTC + ch) * 2;
        float Xr = 0.f, Xi = 0.f;
        if (q == 0) {
            pub_word(incw + me, ar);
            pub_word(incw + me + 1, ai);
        } else {
            pub_word(aggw + me, ar);
            pub_word(aggw + me + 1, ai);
            const cd Lc = cpow(lamd, DCH);
            cd pw = {1.0, 0.0};
            double xr = 0.0, xi = 0.0;
            // look back in windows of LBW predecessors: one round trip per window
            constexpr int LBW = 4;
            int pred = q - 1;
            while (true) {
                unsigned long long iw[LBW][2], aw[LBW][2];
#pragma unroll
                for (int k = 0; k < LBW; ++k) {
                    const int pk = pred - k;
                    iw[k][0] = iw[k][1] = aw[k][0] = aw[k][1] = 0ull;
                    if (pk >= 0) {
                        const size_t pe = (((size_t)st * nq + pk) * DTC + ch) * 2;
                        iw[k][0] = __hip_atomic_load(incw + pe, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        iw[k][1] = __hip_atomic_load(incw + pe + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        aw[k][0] = __hip_atomic_load(aggw + pe, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        aw[k][1] = __hip_atomic_load(aggw + pe + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
                bool done = false;
                int used = 0;
#pragma unroll
                for (int k = 0; k < LBW; ++k) {
                    if (done || used != k || pred - k < 0) continue;
                    const bool inc_ok = (iw[k][0] >> 32) != 0 && (iw[k][1] >> 32) != 0;
                    const bool agg_ok = (aw[k][0] >> 32) != 0 && (aw[k][1] >> 32) != 0;
                    const unsigned long long w0 = inc_ok ? iw[k][0] : aw[k][0], w1 = inc_ok ? iw[k][1] : aw[k][1];
                    if (!inc_ok && !agg_ok) continue;            // not published yet: stop here
                    const double vr = (double)__uint_as_float((uint32_t)w0), vi = (double)__uint_as_float((uint32_t)w1);
                    xr += pw.re * vr - pw.im * vi;
                    xi += pw.re * vi + pw.im * vr;
                    if (inc_ok) {
                        done = true;
                    } else {
                        pw = cmul(pw, Lc);
                        ++used;
                    }
                }
                if (done) break;
                pred -= used;
                if (used == 0) __builtin_amdgcn_s_sleep(1);
            }
            Xr = (float)xr;
            Xi = (float)xi;
            const double ir = (double)ar + (Lc.re * xr - Lc.im * xi), ii = (double)ai + (Lc.re * xi + Lc.im * xr);
            pub_word(incw + me, (float)ir);
            pub_word(incw + me + 1, (float)ii);
        }
        xq[ch] = make_float2(Xr, Xi);
    }
    __syncthreads();
    float yr = pr, yi = pi;
    if (q > 0 && mok) {
        const float2 X = xq[ch];
        const cd Lu = cpow(lamd, (long)usub * DS);
        yr = (float)((double)pr + (Lu.re * X.x - Lu.im * X.y));
        yi = (float)((double)pi + (Lu.re * X.y + Lu.im * X.x));
    }
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const float nr = fmaf(lr, yr, fmaf(-li, yi, bv[s].x));
        const float ni = fmaf(lr, yi, fmaf(li, yr, bv[s].y));
        yr = nr;
        yi = ni;
        const long p = p0 + s;
        if (mok && p < T) {
            const long tau = rev ? (T - 1 - p) : p;
            const v2f o2 = {yr, yi};
            __builtin_nontemporal_store(o2, reinterpret_cast<v2f *>(yout + (((long)b * T + tau) * M + m) * 2));
        }
    }
}

__global__ void k_zero_u64(unsigned long long *p, size_t n) {
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n; e += (size_t)gridDim.x * blockDim.x) p[e] = 0ull;
}

// carries across chunks: one block per (sequence tile, channel); Hillis-Steele over chunks
__global__ __launch_bounds__(256) void k_diag_carry(const float *__restrict__ lam, int conj_lam,
                                                    const float *__restrict__ agg, float *__restrict__ carry,
                                                    int ntile, int M, int nq) {
    __shared__ float2 buf[2][256];
    const int st = blockIdx.x / DTC, ch = blockIdx.x % DTC;
    const int m = (st % ntile) * DTC + ch;
    if (m >= M) return;
    const cd lamd = {(double)lam[2 * m], (double)(conj_lam ? -lam[2 * m + 1] : lam[2 * m + 1])};
    const cd Lc = cpow(lamd, DCH);
    const int tid = threadIdx.x;
    double cr = 0.0, ci = 0.0;          // inclusive value of the previous block's last chunk
    for (int base = 0; base < nq; base += 256) {
        const int q = base + tid;
        float2 v = make_float2(0.f, 0.f);
        if (q < nq) v = reinterpret_cast<const float2 *>(agg)[((long)st * nq + q) * DTC + ch];
        int cur = 0;
        buf[cur][tid] = v;
        __syncthreads();
        cd Ld = Lc;      // Lambda^d
        for (int d = 1; d < 256; d <<= 1) {
            float2 x = buf[cur][tid];
            if (tid >= d) {
                const float2 o = buf[cur][tid - d];
                x.x += (float)(Ld.re * o.x - Ld.im * o.y);
                x.y += (float)(Ld.re * o.y + Ld.im * o.x);
            }
            buf[cur ^ 1][tid] = x;
            __syncthreads();
            cur ^= 1;
            Ld = cmul(Ld, Ld);
        }
        // inclusive I_q (within block) + Lambda^(tid+1) * carry-in from earlier blocks
        const float2 incl = buf[cur][tid];
        const cd Lp = cpow(Lc, tid + 1);
        const double ir = incl.x + (Lp.re * cr - Lp.im * ci), ii = incl.y + (Lp.re * ci + Lp.im * cr);
        // exclusive: X_q = I_{q-1}
        float2 ex;
        if (tid == 0) {
            ex = make_float2((float)cr, (float)ci);
        } else {
            const float2 pin = buf[cur][tid - 1];
            const cd Lq = cpow(Lc, tid);
            ex = make_float2((float)(pin.x + (Lq.re * cr - Lq.im * ci)), (float)(pin.y + (Lq.re * ci + Lq.im * cr)));
        }
        if (q < nq) reinterpret_cast<float2 *>(carry)[((long)st * nq + q) * DTC + ch] = ex;
        __syncthreads();
        // carry for the next block = inclusive value at tid 255
        __shared__ double nxt[2];
        if (tid == 255) {
            nxt[0] = ir;
            nxt[1] = ii;
        }
        __syncthreads();
        cr = nxt[0];
        ci = nxt[1];
        __syncthreads();
    }
}

static bool diag_three_pass() {
    const char *e = getenv("DEER_DIAG_3PASS");
    return e && atoi(e) != 0;
}

size_t diag_scan_ws_bytes(int B, int T, int M) {
    const long ntile = (M + DTC - 1) / DTC;
    const long nq = (T + DCH - 1) / DCH;
    const size_t one = (size_t)B * ntile * nq * DTC * sizeof(float2);
    const size_t three = 2 * ((one + 255) & ~(size_t)255);
    const size_t words = (size_t)B * ntile * nq * DTC * 2 * sizeof(unsigned long long);
    const size_t single = 256 + 2 * ((words + 255) & ~(size_t)255);
    return three > single ? three : single;
}

int launch_diag_scan(bool rev, int B, int T, int M, const float *lam, const float *b, const float *Bc, int K,
                     const float *u, float *y, void *ws, hipStream_t st) {
    const int ntile = (M + DTC - 1) / DTC;
    const int nq = (T + DCH - 1) / DCH;
    const int nblk = B * ntile * nq;
    const int conj_lam = rev ? 1 : 0;
    if (!diag_three_pass()) {
        const size_t nwords = (size_t)B * ntile * nq * DTC * 2;
        const size_t wbytes = (nwords * sizeof(unsigned long long) + 255) & ~(size_t)255;
        unsigned int *ticket = (unsigned int *)ws;
        unsigned long long *aggw = (unsigned long long *)((char *)ws + 256);
        unsigned long long *incw = (unsigned long long *)((char *)ws + 256 + wbytes);
        {
            KTimer _kt("k_zero_u64", st);
            const size_t n = 32 + 2 * wbytes / sizeof(unsigned long long);
            const int grid = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
            hipLaunchKernelGGL(k_zero_u64, dim3(grid), dim3(256), 0, st, (unsigned long long *)ws, n);
        }
        DEER_LAUNCH_CHECK("k_zero_u64");
        {
            KTimer _kt("k_diag_scan_lb", st);
            if (b)
                hipLaunchKernelGGL(k_diag_scan_lb<false>, dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b, Bc, K,
                                   u, rev ? 1 : 0, B, T, M, ntile, nq, ticket, aggw, incw, y);
            else
                hipLaunchKernelGGL(k_diag_scan_lb<true>, dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b, Bc, K,
                                   u, rev ? 1 : 0, B, T, M, ntile, nq, ticket, aggw, incw, y);
        }
        DEER_LAUNCH_CHECK("k_diag_scan_lb");
        return DEER_OK;
    }
    const size_t one = (((size_t)B * ntile * nq * DTC * sizeof(float2)) + 255) & ~(size_t)255;
    float *agg = (float *)ws;
    float *carry = (float *)((char *)ws + one);
    {
        KTimer _kt("k_diag_chunk_reduce", st);
        hipLaunchKernelGGL(k_diag_chunk<false>, dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b, Bc, K, u, rev ? 1 : 0,
                           B, T, M, ntile, nq, agg, (const float *)nullptr, (float *)nullptr);
    }
    DEER_LAUNCH_CHECK("k_diag_chunk<reduce>");
    {
        KTimer _kt("k_diag_carry", st);
        hipLaunchKernelGGL(k_diag_carry, dim3(B * ntile * DTC), dim3(256), 0, st, lam, conj_lam, agg, carry, ntile, M, nq);
    }
    DEER_LAUNCH_CHECK("k_diag_carry");
    {
        KTimer _kt("k_diag_chunk_fixup", st);
        hipLaunchKernelGGL(k_diag_chunk<true>, dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b, Bc, K, u, rev ? 1 : 0,
                           B, T, M, ntile, nq, agg, carry, y);
    }
    DEER_LAUNCH_CHECK("k_diag_chunk<fixup>");
    return DEER_OK;
}

}  // namespace deer

namespace deer {

// Gradients of the diagonal SSM parameters from the adjoint a and the forward states h:
//   dlam_m = sum_{b,t} a_t conj(h_{t-1}),  dBc_{m,k} = sum_{b,t} a_t u_t[k]  (u_t = x_{t-1})
// Pass 1: block = 16 channels x 16 time lanes over a slice of DGT positions -> fp32 partials.
// Pass 2: float64 sum of the partials.
namespace {
constexpr int DGT = 4096;
}

__global__ __launch_bounds__(256) void k_diag_grads_partial(const float *__restrict__ a, const float *__restrict__ h,
                                                            const float *__restrict__ x, int K, int B, int T, int M,
                                                            int ntile, int nsl, float *__restrict__ part) {
    __shared__ float red[16][16][2 + 8];
    const int tl = threadIdx.x >> 4, ch = threadIdx.x & 15;
    const int sl = blockIdx.x % nsl, st = blockIdx.x / nsl;
    const int b = st / ntile, m = (st % ntile) * DTC + ch;
    const bool mok = m < M;
    float acc[2 + 8];
#pragma unroll
    for (int k = 0; k < 10; ++k) acc[k] = 0.f;
    const int t0 = sl * DGT, t1 = min(t0 + DGT, T);
    if (mok) {
        for (int t = t0 + tl; t < t1; t += 16) {
            const float2 av = *reinterpret_cast<const float2 *>(a + (((long)b * T + t) * M + m) * 2);
            if (t > 0) {
                const float2 hv = *reinterpret_cast<const float2 *>(h + (((long)b * T + t - 1) * M + m) * 2);
                acc[0] = fmaf(av.x, hv.x, fmaf(av.y, hv.y, acc[0]));
                acc[1] = fmaf(av.y, hv.x, fmaf(-av.x, hv.y, acc[1]));
            }
            const float *xu = x + ((long)b * (T + 1) + t) * K;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                if (k < K) {
                    const float uk = xu[k];
                    acc[2 + 2 * k] = fmaf(av.x, uk, acc[2 + 2 * k]);
                    acc[3 + 2 * k] = fmaf(av.y, uk, acc[3 + 2 * k]);
                }
        }
    }
#pragma unroll
    for (int k = 0; k < 10; ++k) red[tl][ch][k] = acc[k];
    __syncthreads();
    if (tl == 0 && mok) {
        const int nv = 2 + 2 * K;
        for (int k = 0; k < nv; ++k) {
            float s = 0.f;
            for (int r = 0; r < 16; ++r) s += red[r][ch][k];
            part[(((long)st * nsl + sl) * DTC + ch) * 10 + k] = s;
        }
    }
}

__global__ void k_diag_grads_final(const float *__restrict__ part, int K, int B, int M, int ntile, int nsl,
                                   float *__restrict__ dlam, float *__restrict__ dBc) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;   // (m, k)
    const int nv = 2 + 2 * K;
    if (e >= M * nv) return;
    const int m = e / nv, k = e % nv;
    const int tile = m / DTC, ch = m % DTC;
    double s = 0.0;
    for (int b = 0; b < B; ++b) {
        const int st = b * ntile + tile;
        for (int sl = 0; sl < nsl; ++sl) s += (double)part[(((long)st * nsl + sl) * DTC + ch) * 10 + k];
    }
    if (k < 2) {
        if (dlam) dlam[2 * m + k] = (float)s;
    } else if (dBc) {
        const int kk = (k - 2) / 2, ri = (k - 2) % 2;
        dBc[(m * K + kk) * 2 + ri] = (float)s;
    }
}

size_t diag_grads_ws_bytes(int B, int T, int M) {
    const long ntile = (M + DTC - 1) / DTC;
    const long nsl = (T + DGT - 1) / DGT;
    return (((size_t)B * ntile * nsl * DTC * 10 * sizeof(float)) + 255) & ~(size_t)255;
}

int launch_diag_grads(int B, int T, int M, int K, const float *a, const float *h, const float *x, float *dlam,
                      float *dBc, void *ws, hipStream_t st) {
    const int ntile = (M + DTC - 1) / DTC;
    const int nsl = (T + DGT - 1) / DGT;
    float *part = (float *)ws;
    {
        KTimer _kt("k_diag_grads_partial", st);
        hipLaunchKernelGGL(k_diag_grads_partial, dim3(B * ntile * nsl), dim3(256), 0, st, a, h, x, K, B, T, M, ntile, nsl,
                           part);
    }
    DEER_LAUNCH_CHECK("k_diag_grads_partial");
    const int n = M * (2 + 2 * K);
    {
        KTimer _kt("k_diag_grads_final", st);
        hipLaunchKernelGGL(k_diag_grads_final, dim3((n + 255) / 256), dim3(256), 0, st, part, K, B, M, ntile, nsl, dlam,
                           dBc);
    }
    DEER_LAUNCH_CHECK("k_diag_grads_final");
    return DEER_OK;
}

}  // namespace deer
