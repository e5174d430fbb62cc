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

#include <type_traits>

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
// GRADS (reverse scans only): the adjoint a_tau = y is combined on the fly with the forward
// states h and the inputs x into per-block partial sums of
//   dlam_m = sum a_tau conj(h_{tau-1}),  dBc_{m,k} = sum a_tau x_tau[k]
// (layout part[(k * B * ntile * nq + chain * nq + q) * DTC + ch], k < 2 + 2K); yout may then
// be null (the adjoint itself not stored).
constexpr int DNV = 10;   // 2 + 2 K partial values per channel, K <= 4

// GREAL: b is real [B,T,M] (imaginary part zero), read at 4 bytes per element.
template <bool PROJ, bool GRADS, bool GREAL = false>
__global__ __launch_bounds__(DNW * 64) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_diag_scan_lb(const float *__restrict__ lam, int conj_lam,
                                                          const float *__restrict__ bin, const float *__restrict__ Bc,
                                                          int K, const float *__restrict__ u, int rev, int B, int T,
                                                          int M, int ntile, int nq, unsigned int *__restrict__ ticket,
                                                          unsigned long long *__restrict__ aggw,
                                                          unsigned long long *__restrict__ incw,
                                                          float *__restrict__ yout, const float *__restrict__ hfwd,
                                                          float *__restrict__ part) {
    __shared__ float2 sub[DNW * 4][DTC];
    __shared__ float2 xq[DTC];
    __shared__ float xs[(PROJ || GRADS) ? DCH * 4 : 1];
    __shared__ float red[GRADS ? DNW : 1][DTC][DNV];
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
    if (PROJ || GRADS) {
        // inputs of this chunk staged in LDS with coalesced loads, in position order
        // (PROJ: forward, tau = p; GRADS: reverse, tau = T - 1 - p)
        const long n = (long)DCH * K;
        for (long e = tid; e < n; e += DNW * 64) {
            const long p = (long)q * DCH + e / K;
            const long tau = GRADS ? (T - 1 - p) : p;
            xs[e] = p < T ? u[((long)b * (T + 1) + tau) * K + (e % K)] : 0.f;
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
            if (!PROJ && GREAL) {
                v = make_float2(__builtin_nontemporal_load(bin + ((long)b * T + tau) * M + m), 0.f);
            } else if (!PROJ) {
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
    float acc[DNV];
#pragma unroll
    for (int k = 0; k < DNV; ++k) acc[k] = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const float nr = fmaf(lr, yr, fmaf(-li, yi, bv[s].x));
        const float ni = fmaf(lr, yi, fmaf(li, yr, bv[s].y));
        yr = nr;
        yi = ni;
        const long p = p0 + s;
        if (mok && p < T) {
            const long tau = rev ? (T - 1 - p) : p;
            if (yout) {
                const v2f o2 = {yr, yi};
                __builtin_nontemporal_store(o2, reinterpret_cast<v2f *>(yout + (((long)b * T + tau) * M + m) * 2));
            }
            if (GRADS) {
                if (tau > 0) {
                    const v2f hv = __builtin_nontemporal_load(
                        reinterpret_cast<const v2f *>(hfwd + (((long)b * T + tau - 1) * M + m) * 2));
                    acc[0] = fmaf(yr, hv.x, fmaf(yi, hv.y, acc[0]));
                    acc[1] = fmaf(yi, hv.x, fmaf(-yr, hv.y, acc[1]));
                }
                const float *xu = xs + (long)(usub * DS + s) * K;
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (k < K) {
                        acc[2 + 2 * k] = fmaf(yr, xu[k], acc[2 + 2 * k]);
                        acc[3 + 2 * k] = fmaf(yi, xu[k], acc[3 + 2 * k]);
                    }
            }
        }
    }
    if (GRADS) {
        // sum over the 4 sub-chunks of a wave (lanes ch, ch + 16, ch + 32, ch + 48), then over waves
#pragma unroll
        for (int k = 0; k < DNV; ++k) {
            acc[k] += __shfl_xor(acc[k], 16, 64);
            acc[k] += __shfl_xor(acc[k], 32, 64);
        }
        if (j == 0) {
#pragma unroll
            for (int k = 0; k < DNV; ++k) red[w][ch][k] = acc[k];
        }
        __syncthreads();
        const int nv = 2 + 2 * K;
        if (tid < DTC * nv) {
            const int c2 = tid % DTC, k = tid / DTC;
            float sum = 0.f;
#pragma unroll
            for (int w2 = 0; w2 < DNW; ++w2) sum += red[w2][c2][k];
            part[(((long)k * B * ntile + st) * nq + q) * DTC + c2] = sum;
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

// ---------------------------------------------------------------------------------------
// Forward scan with the input projection fused (y_t = lam y_{t-1} + Bc x_t, y_{-1} = 0, in
// 0-based array positions): the only HBM stream is the output, so the scan is write-bound.
// A wave owns 64 channels (lane = channel: one 512-byte row per step at M = 64) and a
// segment of SEG = 64 * SEG_L consecutive steps that it walks sequentially.  The inputs of
// the segment are loaded once, lane l holding steps SEG_L l .. SEG_L l + SEG_L - 1, and are
// broadcast to the wave with v_readlane as the walk reaches them.  No LDS, no barriers, no
// look-back.
//   k_diag_seg<false>  segment aggregates from zero (reads the inputs only)
//   k_diag_seg_carry   carries across segments in float64 (three-level: groups of segments)
//   k_diag_seg<true>   re-walk of every segment from its carry, y written (plain stores: on this
//                      pattern they sustain ~5% more write bandwidth than non-temporal ones)
// ---------------------------------------------------------------------------------------
constexpr int SEG_L = 8;
constexpr int SEG = 64 * SEG_L;

__device__ __forceinline__ float lane_bcast(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

template <bool WRITE, int K>
__global__ __launch_bounds__(256) void k_diag_seg(const float *__restrict__ lam, const float *__restrict__ Bc,
                                                  const float *__restrict__ u, int B, int T, int M, int nseg,
                                                  int ntile, float2 *__restrict__ agg,
                                                  const float2 *__restrict__ carry, float *__restrict__ y) {
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const long wid = (long)blockIdx.x * 4 + wv;          // (sequence, segment, channel tile)
    if (wid >= (long)B * nseg * ntile) return;
    const int tile = (int)(wid % ntile);
    const long bs = wid / ntile;                          // sequence * nseg + segment
    const int seg = (int)(bs % nseg), b = (int)(bs / nseg);
    const int m = tile * 64 + lane;
    const bool mok = m < M;
    const int t0 = seg * SEG, t1 = min(t0 + SEG, T);
    // inputs of the segment: lane l holds rows t0 + SEG_L l + s, s < SEG_L
    float xv[SEG_L * K];
    {
        const float *xr = u + ((long)b * (T + 1) + t0 + SEG_L * lane) * K;
        const int nrow = min(SEG_L, t1 - t0 - SEG_L * lane);
#pragma unroll
        for (int e = 0; e < SEG_L * K; ++e) xv[e] = e < nrow * K ? xr[e] : 0.f;
    }
    float lr = 0.f, li = 0.f, br[K], bi[K];
#pragma unroll
    for (int k = 0; k < K; ++k) br[k] = bi[k] = 0.f;
    if (mok) {
        lr = lam[2 * m];
        li = lam[2 * m + 1];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            br[k] = Bc[(m * K + k) * 2];
            bi[k] = Bc[(m * K + k) * 2 + 1];
        }
    }
    float hr = 0.f, hi = 0.f;
    if (WRITE && mok) {
        const float2 X = carry[bs * M + m];
        hr = X.x;
        hi = X.y;
    }
    float *yb = y + ((long)b * T + t0) * M * 2 + 2 * m;
    const int ngrp = (t1 - t0 + SEG_L - 1) / SEG_L;
    for (int gq = 0; gq < ngrp; ++gq) {
        const int tb = t0 + gq * SEG_L;
#pragma unroll
        for (int s = 0; s < SEG_L; ++s) {
            float vr = 0.f, vi = 0.f;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float xk = lane_bcast(xv[s * K + k], gq);
                vr = fmaf(br[k], xk, vr);
                vi = fmaf(bi[k], xk, vi);
            }
            if (tb + s < t1) {
                const float nr = fmaf(lr, hr, fmaf(-li, hi, vr));
                const float ni = fmaf(lr, hi, fmaf(li, hr, vi));
                hr = nr;
                hi = ni;
                if (WRITE && mok) {
                    const v2f o2 = {hr, hi};
                    *reinterpret_cast<v2f *>(yb + (long)(tb - t0 + s) * M * 2) = o2;
                }
            }
        }
    }
    if (!WRITE && mok) agg[bs * M + m] = make_float2(hr, hi);
}

// carry[s] = state at the end of segment s - 1:  X_0 = 0,  X_{s+1} = Lambda X_s + A_s,
// Lambda = lam^seglen (conj(lam) for a reverse scan; every segment but the last is full, and
// the last aggregate is not needed).
// Block = (sequence, SEG_CT channels), threads = (group g of CG consecutive segments, channel):
// group aggregates, a sequential pass over the SEG_NG groups, then every group re-walked from
// its carry.  Serial depth 2 CG + SEG_NG instead of nseg; the aggregates of a group are loaded
// SEG_CB at a time (indices clamped to the group, so the loads are unconditional) before the
// dependent float64 updates, so the walks wait on memory once per batch rather than once per
// segment.  16 channels per block and 64 groups: 16 blocks for four sequences of 64 channels,
// and two batches per walk for 2048 segments.
constexpr int SEG_NG = 64;
constexpr int SEG_CT = 16;
constexpr int SEG_CB = 16;

__global__ __launch_bounds__(SEG_NG * SEG_CT) void k_diag_seg_carry(const float *__restrict__ lam, int conj_lam,
                                                                    int seglen, int B, int M, int nseg, int ntile,
                                                                    const float2 *__restrict__ agg,
                                                                    float2 *__restrict__ carry) {
    __shared__ double ga[SEG_NG][SEG_CT][2];
    constexpr int NSUB = 64 / SEG_CT;   // blocks per 64-channel tile
    const int b = blockIdx.x / (ntile * NSUB), rem = blockIdx.x % (ntile * NSUB);
    const int tile = rem / NSUB, sub = rem % NSUB;
    const int ch = threadIdx.x % SEG_CT, grp = threadIdx.x / SEG_CT;
    const int m = tile * 64 + sub * SEG_CT + ch;
    const bool mok = m < M;
    const int CG = (nseg + SEG_NG - 1) / SEG_NG;
    const int s0 = min(grp * CG, nseg), s1 = min(s0 + CG, nseg);
    cd L = {0.0, 0.0};
    if (mok) L = cpow(cd{(double)lam[2 * m], conj_lam ? -(double)lam[2 * m + 1] : (double)lam[2 * m + 1]}, seglen);
    const long base = (long)b * nseg;
    double ar = 0.0, ai = 0.0;
    if (mok) {
        for (int s = s0; s < s1; s += SEG_CB) {
            float2 a[SEG_CB];
#pragma unroll
            for (int j = 0; j < SEG_CB; ++j) a[j] = agg[(base + min(s + j, s1 - 1)) * M + m];
#pragma unroll
            for (int j = 0; j < SEG_CB; ++j) {
                if (s + j < s1) {
                    const double nr = L.re * ar - L.im * ai + (double)a[j].x;
                    const double ni = L.re * ai + L.im * ar + (double)a[j].y;
                    ar = nr;
                    ai = ni;
                }
            }
        }
    }
    ga[grp][ch][0] = ar;
    ga[grp][ch][1] = ai;
    __syncthreads();
    if (grp == 0 && mok) {
        const cd LG = cpow(L, CG);
        double cr = 0.0, ci = 0.0;
        for (int g2 = 0; g2 < SEG_NG; ++g2) {
            const double xr = ga[g2][ch][0], xi = ga[g2][ch][1];
            ga[g2][ch][0] = cr;
            ga[g2][ch][1] = ci;
            const double nr = LG.re * cr - LG.im * ci + xr;
            const double ni = LG.re * ci + LG.im * cr + xi;
            cr = nr;
            ci = ni;
        }
    }
    __syncthreads();
    if (!mok) return;
    double xr = ga[grp][ch][0], xi = ga[grp][ch][1];
    for (int s = s0; s < s1; s += SEG_CB) {
        float2 a[SEG_CB];
#pragma unroll
        for (int j = 0; j < SEG_CB; ++j) a[j] = agg[(base + min(s + j, s1 - 1)) * M + m];
#pragma unroll
        for (int j = 0; j < SEG_CB; ++j) {
            if (s + j < s1) {
                carry[(base + s + j) * M + m] = make_float2((float)xr, (float)xi);
                const double nr = L.re * xr - L.im * xi + (double)a[j].x;
                const double ni = L.re * xi + L.im * xr + (double)a[j].y;
                xr = nr;
                xi = ni;
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// Segment aggregates of the forward scan on the matrix cores (M <= 64, K <= 4 inputs).  The
// state a full segment [t0, t0 + 512) reaches from zero is, per channel,
//   A = sum_{a < 8} lam^{64 (7 - a)} sum_{j < K} Bc_j R_{a,j},
//   R_{a,j} = sum_{k < 64} lam^{63 - k} u_{t0 + 64 a + k, j},
// and R for the 64 channels (real parts in rows 0..63, imaginary parts in rows 64..127) and
// the 32 columns (a, j) is one [128 x 64] x [64 x 32] product: A operand = the powers
// lam^{63 - k} (LDS, formed once per block in float64), B operand = the segment's inputs
// (registers).  The k order is permuted as in the read-out (k-step
// (jj, q) of lane group g is k = 16 jj + 4 g + q) so that one 16-byte LDS read gives four
// k-steps of either operand.  The epilogue multiplies every column by lam^{64 (7 - a)} Bc_j
// and sums the 16 columns of a tile across its lanes.  A wave takes one segment at a time; a
// partial last segment gets an aggregate that is never used (the carries stop before it).
// ---------------------------------------------------------------------------------------
constexpr int AGW = 4;        // waves (segments in flight) per block

// sum over the 16 lanes of a DPP row, in every lane of it (row rotations by 8, 4, 2, 1)
__device__ __forceinline__ float row16_sum(float v) {
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xF, 0xF, true));
    return v;
}
constexpr int AQS = 68;       // LDS row stride of the powers and of the transposed inputs

__global__ __launch_bounds__(AGW * 64) void k_diag_seg_agg(const float *__restrict__ lam, const float *__restrict__ Bc,
                                                           const float *__restrict__ u, int B, int T, int M, int K,
                                                           int nseg, float2 *__restrict__ agg) {
    static_assert(SEG == 512, "8 blocks of 64 steps per segment");
    __shared__ __align__(16) float qs[128][AQS];           // lam^{63-k}: re rows 0..63, im rows 64..127
    __shared__ float2 pw[64][8], bcs[64][4];                // lam^{64 (7 - a)}, Bc_j
    const int tid = threadIdx.x;
    // powers in float64: a thread takes 8 consecutive k of one channel (one power, then 7 products)
    for (int e = tid; e < 64 * 8; e += AGW * 64) {
        const int ch = e / 8, kb = e % 8;
        const cd l = ch < M ? cd{(double)lam[2 * ch], (double)lam[2 * ch + 1]} : cd{0.0, 0.0};
        cd p = cpow(l, 56 - 8 * kb);   // lam^{63 - k} for k = 8 kb + 7
        for (int k = 8 * kb + 7; k >= 8 * kb; --k) {
            qs[ch][k] = (float)p.re;
            qs[64 + ch][k] = (float)p.im;
            p = cmul(p, l);
        }
    }
    if (tid < 64) {
        const int ch = tid;
        const cd l = ch < M ? cd{(double)lam[2 * ch], (double)lam[2 * ch + 1]} : cd{0.0, 0.0};
        const cd l64 = cpow(l, 64);
        cd p = {1.0, 0.0};
        for (int a = 7; a >= 0; --a) {   // lam^{64 (7 - a)}
            pw[ch][a] = make_float2((float)p.re, (float)p.im);
            p = cmul(p, l64);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            bcs[ch][j] = (ch < M && j < K) ? make_float2(Bc[(ch * K + j) * 2], Bc[(ch * K + j) * 2 + 1])
                                           : make_float2(0.f, 0.f);
    }
    __syncthreads();
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, c = lane & 15;
    const long total = (long)B * nseg;
    const long stride = (long)gridDim.x * AGW;
    // B operands of a segment straight from the inputs: k-step (jj, q) of lane (g, c) in column
    // tile J is input j = c % 4 of step t0 + 64 a + 16 jj + 4 g + q, a = 4 J + c / 4 (zero past the
    // sequence and for j >= K), loaded into registers at the start of the segment (the other
    // waves of the CU cover the wait)
    float nb[2][4][4];
    const int jin = c & 3;
    auto fetch = [&](long sid) {
        const bool in = sid < total;
        const int b = in ? (int)(sid / nseg) : 0, seg = in ? (int)(sid % nseg) : 0;
        const int t0 = seg * SEG;
        const float *ub = u + (long)b * (T + 1) * K;
#pragma unroll
        for (int J = 0; J < 2; ++J)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int t = t0 + 64 * (4 * J + (c >> 2)) + 16 * jj + 4 * g + q;
                    const bool ok = in && t < T && jin < K;
                    nb[J][jj][q] = ok ? ub[(long)t * K + jin] : 0.f;
                }
    };
    for (long sid = (long)blockIdx.x * AGW + wv; sid < total; sid += stride) {
        fetch(sid);
        // the powers are read from LDS k-block by k-block inside the loop (kept out of registers
        // across segments, which leaves room for three waves per SIMD)
        asm volatile("" ::: "memory");
        v4f acc[8][2];
#pragma unroll
        for (int I = 0; I < 8; ++I) acc[I][0] = acc[I][1] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            float4 aq[8], bq[2];
#pragma unroll
            for (int I = 0; I < 8; ++I) aq[I] = *reinterpret_cast<const float4 *>(&qs[16 * I + c][16 * jj + 4 * g]);
#pragma unroll
            for (int J = 0; J < 2; ++J) bq[J] = make_float4(nb[J][jj][0], nb[J][jj][1], nb[J][jj][2], nb[J][jj][3]);
            // 16 independent accumulators between two products into the same one
#pragma unroll
            for (int J = 0; J < 2; ++J)
#pragma unroll
                for (int I = 0; I < 8; ++I) acc[I][J] = mfma16x16x4(aq[I].x, bq[J].x, acc[I][J]);
#pragma unroll
            for (int J = 0; J < 2; ++J)
#pragma unroll
                for (int I = 0; I < 8; ++I) acc[I][J] = mfma16x16x4(aq[I].y, bq[J].y, acc[I][J]);
#pragma unroll
            for (int J = 0; J < 2; ++J)
#pragma unroll
                for (int I = 0; I < 8; ++I) acc[I][J] = mfma16x16x4(aq[I].z, bq[J].z, acc[I][J]);
#pragma unroll
            for (int J = 0; J < 2; ++J)
#pragma unroll
                for (int I = 0; I < 8; ++I) acc[I][J] = mfma16x16x4(aq[I].w, bq[J].w, acc[I][J]);
        }
        // epilogue: lane (g, c) holds rows 16 I + 4 g + r (channel 16 (I % 4) + 4 g + r, real part
        // for I < 4, imaginary for I >= 4) of columns 16 J + c = (a = 4 J + c / 4, j = c % 4)
        float sr[4][4], si[4][4];
#pragma unroll
        for (int I = 0; I < 4; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ch = 16 * I + 4 * g + r;
                float xr = 0.f, xi = 0.f;
#pragma unroll
                for (int J = 0; J < 2; ++J) {
                    const float2 p = pw[ch][4 * J + (c >> 2)], q = bcs[ch][c & 3];
                    const float kr = p.x * q.x - p.y * q.y, ki = p.x * q.y + p.y * q.x;   // lam^{64 (7-a)} Bc_j
                    const float Rr = acc[I][J][r], Ri = acc[I + 4][J][r];
                    xr = fmaf(kr, Rr, fmaf(-ki, Ri, xr));
                    xi = fmaf(kr, Ri, fmaf(ki, Rr, xi));
                }
                sr[I][r] = xr;
                si[I][r] = xi;
            }
#pragma unroll
        for (int I = 0; I < 4; ++I)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sr[I][r] = row16_sum(sr[I][r]);
                si[I][r] = row16_sum(si[I][r]);
            }
        if (c == 0) {
#pragma unroll
            for (int I = 0; I < 4; ++I)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int ch = 16 * I + 4 * g + r;
                    if (ch < M) agg[sid * M + ch] = make_float2(sr[I][r], si[I][r]);
                }
        }
    }
}

static bool diag_seg_enabled() {
    const char *e = getenv("DEER_DIAG_SEG");
    return !e || atoi(e) != 0;
}

// segment aggregates on the matrix cores (DEER_DIAG_AGG_MFMA=0: the lane-per-channel walk)
static bool diag_agg_mfma() {
    const char *e = getenv("DEER_DIAG_AGG_MFMA");
    return !e || atoi(e) != 0;
}

static size_t diag_seg_ws_bytes(int B, int T, int M) {
    const size_t nseg = (T + SEG - 1) / SEG;
    const size_t one = ((size_t)B * nseg * M * sizeof(float2) + 255) & ~(size_t)255;
    return 2 * one;
}

static int launch_diag_seg(int B, int T, int M, const float *lam, const float *Bc, int K, const float *u, float *y,
                           void *ws, hipStream_t st) {
    const int nseg = (T + SEG - 1) / SEG;
    const int ntile = (M + 63) / 64;
    const size_t one = ((size_t)B * nseg * M * sizeof(float2) + 255) & ~(size_t)255;
    float2 *agg = (float2 *)ws;
    float2 *carry = (float2 *)((char *)ws + one);
    const long waves = (long)B * nseg * ntile;
    const int grid = (int)((waves + 3) / 4);
#define SEGK(WR, KV, A, C, Y) \
    hipLaunchKernelGGL((k_diag_seg<WR, KV>), dim3(grid), dim3(256), 0, st, lam, Bc, u, B, T, M, nseg, ntile, A, C, Y)
#define SEGALL(WR, A, C, Y)                  \
    switch (K) {                             \
        case 1: SEGK(WR, 1, A, C, Y); break; \
        case 2: SEGK(WR, 2, A, C, Y); break; \
        case 3: SEGK(WR, 3, A, C, Y); break; \
        default: SEGK(WR, 4, A, C, Y); break; \
    }
    if (M <= 64 && K <= 4 && diag_agg_mfma()) {
        // segment aggregates on the matrix cores: a few blocks per CU, each forming the powers once
        const long segs = (long)B * nseg;
        const long want = (segs + AGW - 1) / AGW;
        const int gridm = (int)(want < 768 ? want : 768);   // three blocks per CU
        KTimer _kt("k_diag_seg_reduce", st);
        hipLaunchKernelGGL(k_diag_seg_agg, dim3(gridm), dim3(AGW * 64), 0, st, lam, Bc, u, B, T, M, K, nseg, agg);
    } else {
        KTimer _kt("k_diag_seg_reduce", st);
        SEGALL(false, agg, (const float2 *)nullptr, (float *)nullptr)
    }
    DEER_LAUNCH_CHECK("k_diag_seg<reduce>");
    {
        KTimer _kt("k_diag_seg_carry", st);
        hipLaunchKernelGGL(k_diag_seg_carry, dim3(B * ntile * (64 / SEG_CT)), dim3(SEG_NG * SEG_CT), 0, st, lam, 0, SEG, B,
                           M, nseg, ntile,
                           (const float2 *)agg, carry);
    }
    DEER_LAUNCH_CHECK("k_diag_seg_carry");
    {
        KTimer _kt("k_diag_seg_write", st);
        SEGALL(true, (float2 *)nullptr, (const float2 *)carry, y)
    }
#undef SEGALL
#undef SEGK
    DEER_LAUNCH_CHECK("k_diag_seg<write>");
    return DEER_OK;
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
    size_t need = three > single ? three : single;
    const size_t seg = diag_seg_ws_bytes(B, T, M);
    return need > seg ? need : seg;
}

int launch_diag_scan(bool rev, int B, int T, int M, const float *lam, const float *b, const float *Bc, int K,
                     const float *u, float *y, void *ws, hipStream_t st, int conj) {
    const int ntile = (M + DTC - 1) / DTC;
    const int nq = (T + DCH - 1) / DCH;
    const int nblk = B * ntile * nq;
    const int conj_lam = conj < 0 ? (rev ? 1 : 0) : (conj ? 1 : 0);
    if (!b && !rev && conj_lam == 0 && diag_seg_enabled()) return launch_diag_seg(B, T, M, lam, Bc, K, u, y, ws, st);
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
                hipLaunchKernelGGL((k_diag_scan_lb<false, false>), dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b,
                                   Bc, K, u, rev ? 1 : 0, B, T, M, ntile, nq, ticket, aggw, incw, y,
                                   (const float *)nullptr, (float *)nullptr);
            else
                hipLaunchKernelGGL((k_diag_scan_lb<true, false>), dim3(nblk), dim3(DNW * 64), 0, st, lam, conj_lam, b,
                                   Bc, K, u, rev ? 1 : 0, B, T, M, ntile, nq, ticket, aggw, incw, y,
                                   (const float *)nullptr, (float *)nullptr);
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

// float64 sums of the fused-scan partials.  Stage 1: block = (channel tile, value k, slice of
// the B * nq chunk rows), lanes (row r, channel ch); stage 2 sums the slices.
constexpr int DGS = 64;   // slices

__global__ __launch_bounds__(256) void k_diag_grads_sum1(const float *__restrict__ part, int B, int ntile, int nq,
                                                         double *__restrict__ part2) {
    __shared__ double red[16][DTC];
    const int sl = blockIdx.x % DGS, tk = blockIdx.x / DGS;   // tk = k * ntile + tile
    const int tile = tk % ntile, k = tk / ntile;
    const int tid = threadIdx.x, r = tid / DTC, ch = tid % DTC;
    const long rows = (long)B * nq;
    const long r0 = rows * sl / DGS, r1 = rows * (sl + 1) / DGS;
    double s = 0.0;
    for (long row = r0 + r; row < r1; row += 16) {
        const long bb = row / nq, q = row % nq;
        s += (double)part[(((long)k * B * ntile + bb * ntile + tile) * nq + q) * DTC + ch];
    }
    red[r][ch] = s;
    __syncthreads();
    if (tid < DTC) {
        double t = 0.0;
        for (int r2 = 0; r2 < 16; ++r2) t += red[r2][tid];
        part2[((long)tk * DGS + sl) * DTC + tid] = t;
    }
}

__global__ __launch_bounds__(64) void k_diag_grads_sum2(const double *__restrict__ part2, int K, int M, int ntile,
                                                        float *__restrict__ dlam, float *__restrict__ dBc) {
    const int e = blockIdx.x * 64 + threadIdx.x;   // (k, m)
    if (e >= (2 + 2 * K) * ntile * DTC) return;
    const int ch = e % DTC, tk = e / DTC;
    const int tile = tk % ntile, k = tk / ntile;
    const int m = tile * DTC + ch;
    if (m >= M) return;
    double t = 0.0;
    for (int sl = 0; sl < DGS; ++sl) t += part2[((long)tk * DGS + sl) * DTC + ch];
    if (k < 2) {
        if (dlam) dlam[2 * m + k] = (float)t;
    } else if (dBc) {
        const int kk = (k - 2) / 2, ri = (k - 2) % 2;
        dBc[(m * K + kk) * 2 + ri] = (float)t;
    }
}

// ---------------------------------------------------------------------------------------
// Reverse scan of a cotangent g with the parameter gradients, for callers that keep the
// gradients only (the adjoint itself is not stored): one read of g and of the forward states
// h, in whole rows (lane = channel, 64 channels per wave).
//   a_tau = conj(lam) a_{tau+1} + g_tau  (a_T = 0),
//   dlam_m = sum_{tau >= 1} a_tau conj(h_{tau-1}),   dBc_{m,k} = sum_tau a_tau x_tau[k].
// Logical positions p = T - 1 - tau; segment r of a sequence covers p in [r S, min(r S + S, T)).
// A wave walks its segment from a zero state, giving the local adjoint y_p; the adjoint itself
// is y_p + c_p X_r with c_p = conj(lam)^(p - r S + 1) and X_r the adjoint at p = r S - 1 (the
// carry).  That is linear in X_r, so the wave accumulates
//   P1 = sum y conj(h),  P2 = sum c conj(h),  Q1_k = sum y x[k],  Q2_k = sum c x[k]
// and, once k_diag_seg_carry has formed every X_r from the segment aggregates (y at the
// segment's last position), k_diag_rseg_sum adds dlam = sum_r P1 + X_r P2 and
// dBc_k = sum_r Q1_k + X_r Q2_k.  c restarts from a float64 power every RSUB steps; the sums
// run in float32 per 64 steps and are then added into float32 segment totals.
// The inputs x of 64 consecutive steps sit one per lane and reach the wave through
// v_readlane.  Register batches of RSUB steps: the next batch's loads are issued before the
// current batch is walked.
// part layout: part[(v B nseg + b nseg + r) M + m], v < 4 + 4 K (P1 re, im, P2 re, im, then
// per k: Q1 re, im, Q2 re, im); agg[(b nseg + r) M + m].
// ---------------------------------------------------------------------------------------
constexpr int RSUB = 8;

template <int K, bool GREAL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_diag_rseg(const float *__restrict__ lam, const float *__restrict__ g,
                                                   const float *__restrict__ h, const float *__restrict__ x, int B,
                                                   int T, int M, int nseg, int S, int ntile,
                                                   float2 *__restrict__ agg, float *__restrict__ part) {
    constexpr int NP = 4 + 4 * K;
    constexpr int GW = GREAL ? 1 : 2;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const long wid = (long)blockIdx.x * 4 + wv;   // (sequence, segment, channel tile)
    if (wid >= (long)B * nseg * ntile) return;
    const int tile = (int)(wid % ntile);
    const long bs = wid / ntile;
    const int r = (int)(bs % nseg), b = (int)(bs / nseg);
    const int m = tile * 64 + lane;
    const bool mok = m < M;
    const int p0 = r * S, p1 = min(p0 + S, T);
    float lr = 0.f, li = 0.f;
    if (mok) {
        lr = lam[2 * m];
        li = -lam[2 * m + 1];
    }
    const cd lc = {(double)lr, (double)li};
    const cd lsub = cpow(lc, RSUB);
    cd cb = lc;   // c at the first step of the current batch
    // g rows tau and h rows tau - 1 through buffer resources based at row tau_lo of sequence b:
    // one lane offset for every load (>= 2^31 outside the resource for lanes past M: those loads
    // return 0) and the row offset in an SGPR
    const int tau_lo = max(T - p1 - 1, 0);
    const auto rg = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(g + ((long)b * T + tau_lo) * M * GW),
                                                      (short)0, 0x7fffffff, 0x00020000);
    const auto rh = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(h + ((long)b * T + tau_lo) * M * 2),
                                                      (short)0, 0x7fffffff, 0x00020000);
    const int vog = mok ? m * 4 * GW : (int)0x80000000, voh = mok ? m * 8 : (int)0x80000000;
    const float *xb = x + (long)b * (T + 1) * K;

    float gc[RSUB * GW], hc[RSUB * 2], gn[RSUB * GW], hn[RSUB * 2];
    float xv[K], xn[K];
    // a batch is guarded when it is partial or holds tau = 0 (no h row before it): then every
    // load is conditional; other batches load unconditionally
    auto load_batch = [&](int pb, float *gd, float *hd, auto guard) {
        constexpr bool GUARD = decltype(guard)::value;
        const int nv = min(RSUB, p1 - pb);
#pragma unroll
        for (int s = 0; s < RSUB; ++s) {
            const int tau = T - 1 - (pb + s);
            const int rowo = (tau - tau_lo) * M;
            float g0 = 0.f, g1 = 0.f, h0 = 0.f, h1 = 0.f;
            if (!GUARD || s < nv) {
                if (GREAL) {
                    g0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rg, vog, rowo * 4, 0));
                } else {
                    const v2f t2 = __builtin_bit_cast(v2f, __builtin_amdgcn_raw_buffer_load_b64(rg, vog, rowo * 8, 0));
                    g0 = t2.x;
                    g1 = t2.y;
                }
                if (!GUARD || tau > 0) {
                    const v2f t2 =
                        __builtin_bit_cast(v2f, __builtin_amdgcn_raw_buffer_load_b64(rh, voh, rowo * 8 - M * 8, 0));
                    h0 = t2.x;
                    h1 = t2.y;
                }
            }
            gd[s * GW] = g0;
            if (!GREAL) gd[s * GW + 1] = g1;
            hd[2 * s] = h0;
            hd[2 * s + 1] = h1;
        }
    };
    auto guarded = [&](int pb) { return pb + RSUB >= T || pb + RSUB > p1; };
    auto load_x = [&](int pg, float *xd) {
        const int p = pg + lane;
#pragma unroll
        for (int k = 0; k < K; ++k) xd[k] = p < p1 ? xb[((long)T - 1 - p) * K + k] : 0.f;
    };
    float yr = 0.f, yi = 0.f;
    // segment totals in LDS (each lane its own words, no barrier), float32 sums of 64 steps in
    // registers
    __shared__ float tot[4][4 + 4 * K][64];
    float acc[4 + 4 * K];
#pragma unroll
    for (int v = 0; v < NP; ++v) {
        tot[wv][v][lane] = 0.f;
        acc[v] = 0.f;
    }
    auto walk = [&](int pb, auto guard) {
        constexpr bool GUARD = decltype(guard)::value;
        const int q = pb - p0;
        const int nv = min(RSUB, p1 - pb);
        float cr = (float)cb.re, ci = (float)cb.im;
#pragma unroll
        for (int s = 0; s < RSUB; ++s) {
            if (!GUARD || s < nv) {
                const float g0 = gc[s * GW], g1 = GREAL ? 0.f : gc[s * GW + 1];
                const float nr = fmaf(lr, yr, fmaf(-li, yi, g0));
                const float ni = fmaf(lr, yi, fmaf(li, yr, g1));
                yr = nr;
                yi = ni;
                const float h0 = hc[2 * s], h1 = hc[2 * s + 1];
                acc[0] = fmaf(yr, h0, fmaf(yi, h1, acc[0]));
                acc[1] = fmaf(yi, h0, fmaf(-yr, h1, acc[1]));
                acc[2] = fmaf(cr, h0, fmaf(ci, h1, acc[2]));
                acc[3] = fmaf(ci, h0, fmaf(-cr, h1, acc[3]));
                const int xl = (q & 63) + s;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const float xk = lane_bcast(xv[k], xl);
                    acc[4 + 4 * k] = fmaf(yr, xk, acc[4 + 4 * k]);
                    acc[5 + 4 * k] = fmaf(yi, xk, acc[5 + 4 * k]);
                    acc[6 + 4 * k] = fmaf(cr, xk, acc[6 + 4 * k]);
                    acc[7 + 4 * k] = fmaf(ci, xk, acc[7 + 4 * k]);
                }
                const float tr = cr * lr - ci * li;
                ci = cr * li + ci * lr;
                cr = tr;
            }
        }
    };
    using GOFF = std::integral_constant<bool, false>;
    using GON = std::integral_constant<bool, true>;
    load_x(p0, xv);
    if (guarded(p0)) load_batch(p0, gc, hc, GON{});
    else load_batch(p0, gc, hc, GOFF{});
    for (int pb = p0; pb < p1; pb += RSUB) {
        const int q = pb - p0;
        const bool more = pb + RSUB < p1;
        const bool newgrp = ((q + RSUB) & 63) == 0;
        if (more) {
            if (guarded(pb + RSUB)) load_batch(pb + RSUB, gn, hn, GON{});
            else load_batch(pb + RSUB, gn, hn, GOFF{});
            if (newgrp) load_x(pb + RSUB, xn);
        }
        if (guarded(pb)) walk(pb, GON{});
        else walk(pb, GOFF{});
        cb = cmul(cb, lsub);
        if (newgrp || !more) {
#pragma unroll
            for (int v = 0; v < NP; ++v) {
                tot[wv][v][lane] += acc[v];
                acc[v] = 0.f;
            }
        }
        if (more) {
#pragma unroll
            for (int e = 0; e < RSUB * GW; ++e) gc[e] = gn[e];
#pragma unroll
            for (int e = 0; e < RSUB * 2; ++e) hc[e] = hn[e];
            if (newgrp) {
#pragma unroll
                for (int k = 0; k < K; ++k) xv[k] = xn[k];
            }
        }
    }
    if (!mok) return;
    agg[bs * M + m] = make_float2(yr, yi);
    const long vs = (long)B * nseg * M;
#pragma unroll
    for (int v = 0; v < NP; ++v) part[v * vs + bs * M + m] = tot[wv][v][lane];
}

// float64 sums of the segment terms: dlam = sum_r P1 + X_r P2, dBc_k = sum_r Q1_k + X_r Q2_k.
// Block = (64-channel tile, slice of the B nseg segment rows), 16 row lanes x 64 channels;
// a thread loads RSR rows at a time (indices clamped to the slice, loads unconditional) before
// adding them.  The slice sums go to part2 in the layout k_diag_grads_sum2 reads (value,
// 16-channel tile, slice, channel).
constexpr int RSR = 4;

template <int K>
__global__ __launch_bounds__(1024) void k_diag_rseg_sum(const float2 *__restrict__ carry, const float *__restrict__ part,
                                                        long rows, int M, int ntile16, double *__restrict__ part2) {
    constexpr int NV = 2 + 2 * K;
    constexpr int NP = 4 + 4 * K;
    __shared__ double red[16][NV][64];
    const int sl = blockIdx.x % DGS, tile = blockIdx.x / DGS;
    const int rl = threadIdx.x >> 6, ch = threadIdx.x & 63;
    const int m = tile * 64 + ch;
    const bool mok = m < M;
    const long r0 = rows * sl / DGS, r1 = rows * (sl + 1) / DGS;
    const long vs = rows * M;
    double acc[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) acc[v] = 0.0;
    if (mok && r1 > r0) {
        for (long rb = r0 + rl; rb < r1; rb += 16 * RSR) {
            float2 X[RSR];
            float pv[RSR][NP];
#pragma unroll
            for (int j = 0; j < RSR; ++j) {
                const long row = min(rb + 16 * j, r1 - 1);
                X[j] = carry[row * M + m];
#pragma unroll
                for (int v = 0; v < NP; ++v) pv[j][v] = part[v * vs + row * M + m];
            }
#pragma unroll
            for (int j = 0; j < RSR; ++j) {
                if (rb + 16 * j < r1) {
                    const double xr = X[j].x, xi = X[j].y;
                    double pr = pv[j][2], pi = pv[j][3];
                    acc[0] += (double)pv[j][0] + (xr * pr - xi * pi);
                    acc[1] += (double)pv[j][1] + (xr * pi + xi * pr);
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        pr = pv[j][6 + 4 * k];
                        pi = pv[j][7 + 4 * k];
                        acc[2 + 2 * k] += (double)pv[j][4 + 4 * k] + (xr * pr - xi * pi);
                        acc[3 + 2 * k] += (double)pv[j][5 + 4 * k] + (xr * pi + xi * pr);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) red[rl][v][ch] = acc[v];
    __syncthreads();
    if (rl < NV && mok) {
        double t = 0.0;
#pragma unroll
        for (int r2 = 0; r2 < 16; ++r2) t += red[r2][rl][ch];
        part2[(((long)rl * ntile16 + m / 16) * DGS + sl) * 16 + m % 16] = t;
    }
}

// segment length of the reverse walk: whole 64-step groups, long enough to keep the carry
// pass short, short enough for ~4096 waves
static int diag_rseg_len(int B, int T, int M) {
    const char *e = getenv("DEER_DIAG_RSEG");
    if (e && atoi(e) >= 64) return (atoi(e) / 64) * 64;
    const long ntile = (M + 63) / 64;
    int S = 1024;
    while (S > 128 && (long)B * ((T + S - 1) / S) * ntile < 4096) S /= 2;
    return S;
}

static bool diag_rseg_enabled() {
    const char *e = getenv("DEER_DIAG_RSEG");
    return !e || atoi(e) != 0;
}

static size_t diag_rseg_ws_bytes(int B, int T, int M, int K) {
    const int S = diag_rseg_len(B, T, M);
    const size_t nseg = (T + S - 1) / S;
    const size_t one = ((size_t)B * nseg * M * sizeof(float2) + 255) & ~(size_t)255;
    const size_t parts = (((size_t)(4 + 4 * K) * B * nseg * M * sizeof(float)) + 255) & ~(size_t)255;
    const size_t ntile16 = (M + 15) / 16;
    const size_t parts2 = (size_t)(2 + 2 * K) * ntile16 * DGS * 16 * sizeof(double);
    return 2 * one + parts + parts2;
}

size_t diag_adjoint_ws_bytes(int B, int T, int M, int K) {
    const long ntile = (M + DTC - 1) / DTC;
    const long nq = (T + DCH - 1) / DCH;
    const size_t words = (size_t)B * ntile * nq * DTC * 2 * sizeof(unsigned long long);
    const size_t parts = (size_t)(2 + 2 * K) * B * ntile * nq * DTC * sizeof(float);
    const size_t parts2 = (size_t)(2 + 2 * K) * ntile * DGS * DTC * sizeof(double);
    const size_t lb = 256 + 2 * ((words + 255) & ~(size_t)255) + ((parts + 255) & ~(size_t)255) + parts2;
    const size_t rs = diag_rseg_ws_bytes(B, T, M, K);
    return lb > rs ? lb : rs;
}

// Reverse scan of the cotangent g with the parameter gradients fused (dlam, dBc may be
// null; lam_out may be null).
int launch_diag_adjoint(int B, int T, int M, int K, const float *lam, const float *g, bool g_real, const float *h,
                        const float *x, float *lam_out, float *dlam, float *dBc, void *ws, hipStream_t st) {
    const bool grads = dlam || dBc;
    if (grads && !lam_out && K >= 1 && K <= 4 && diag_rseg_enabled()) {
        // gradients only: one segment walk over g and h, carries of the segment aggregates,
        // then the segment terms combined with their carries
        const int S = diag_rseg_len(B, T, M);
        const int nseg = (T + S - 1) / S;
        const int nt64 = (M + 63) / 64, nt16 = (M + 15) / 16;
        const size_t one = ((size_t)B * nseg * M * sizeof(float2) + 255) & ~(size_t)255;
        const size_t parts = (((size_t)(4 + 4 * K) * B * nseg * M * sizeof(float)) + 255) & ~(size_t)255;
        float2 *agg = (float2 *)ws;
        float2 *carry = (float2 *)((char *)ws + one);
        float *part = (float *)((char *)ws + 2 * one);
        double *part2 = (double *)((char *)part + parts);
        const long waves = (long)B * nseg * nt64;
        const int grid = (int)((waves + 3) / 4);
        {
            KTimer _kt("k_diag_rseg", st);
#define RSEGK(KV, RE)                                                                                              \
    hipLaunchKernelGGL((k_diag_rseg<KV, RE>), dim3(grid), dim3(256), 0, st, lam, g, h, x, B, T, M, nseg, S, nt64, agg, \
                       part)
#define RSEGALL(RE)                        \
    switch (K) {                           \
        case 1: RSEGK(1, RE); break;       \
        case 2: RSEGK(2, RE); break;       \
        case 3: RSEGK(3, RE); break;       \
        default: RSEGK(4, RE); break;      \
    }
            if (g_real) {
                RSEGALL(true)
            } else {
                RSEGALL(false)
            }
#undef RSEGALL
#undef RSEGK
        }
        DEER_LAUNCH_CHECK("k_diag_rseg");
        {
            KTimer _kt("k_diag_seg_carry_rev", st);
            hipLaunchKernelGGL(k_diag_seg_carry, dim3(B * nt64 * (64 / SEG_CT)), dim3(SEG_NG * SEG_CT), 0, st, lam, 1, S,
                               B, M, nseg, nt64,
                               (const float2 *)agg, carry);
        }
        DEER_LAUNCH_CHECK("k_diag_seg_carry<rev>");
        {
            KTimer _kt("k_diag_grads_sum", st);
            const long rows = (long)B * nseg;
            switch (K) {
                case 1: hipLaunchKernelGGL(k_diag_rseg_sum<1>, dim3(nt64 * DGS), dim3(1024), 0, st, (const float2 *)carry, (const float *)part, rows, M, nt16, part2); break;
                case 2: hipLaunchKernelGGL(k_diag_rseg_sum<2>, dim3(nt64 * DGS), dim3(1024), 0, st, (const float2 *)carry, (const float *)part, rows, M, nt16, part2); break;
                case 3: hipLaunchKernelGGL(k_diag_rseg_sum<3>, dim3(nt64 * DGS), dim3(1024), 0, st, (const float2 *)carry, (const float *)part, rows, M, nt16, part2); break;
                default: hipLaunchKernelGGL(k_diag_rseg_sum<4>, dim3(nt64 * DGS), dim3(1024), 0, st, (const float2 *)carry, (const float *)part, rows, M, nt16, part2); break;
            }
            const int nv = 2 + 2 * K;
            hipLaunchKernelGGL(k_diag_grads_sum2, dim3((nv * nt16 * DTC + 63) / 64), dim3(64), 0, st,
                               (const double *)part2, K, M, nt16, dlam, dBc);
        }
        DEER_LAUNCH_CHECK("k_diag_rseg_sum");
        return DEER_OK;
    }
    const int ntile = (M + DTC - 1) / DTC;
    const int nq = (T + DCH - 1) / DCH;
    const int nblk = B * ntile * nq;
    const size_t nwords = (size_t)B * ntile * nq * DTC * 2;
    const size_t wbytes = (nwords * sizeof(unsigned long long) + 255) & ~(size_t)255;
    unsigned int *ticket = (unsigned int *)ws;
    unsigned long long *aggw = (unsigned long long *)((char *)ws + 256);
    unsigned long long *incw = (unsigned long long *)((char *)ws + 256 + wbytes);
    float *part = (float *)((char *)ws + 256 + 2 * wbytes);
    const size_t pbytes = ((size_t)(2 + 2 * K) * B * ntile * nq * DTC * sizeof(float) + 255) & ~(size_t)255;
    double *part2 = (double *)((char *)part + pbytes);
    {
        KTimer _kt("k_zero_u64", st);
        const size_t n = 32 + 2 * wbytes / sizeof(unsigned long long);
        const int grid = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
        hipLaunchKernelGGL(k_zero_u64, dim3(grid), dim3(256), 0, st, (unsigned long long *)ws, n);
    }
    DEER_LAUNCH_CHECK("k_zero_u64");
    {
        KTimer _kt(grads ? "k_diag_scan_lb_grads" : "k_diag_scan_lb", st);
#define LBA(GR, RE, HP, PP)                                                                                        \
    hipLaunchKernelGGL((k_diag_scan_lb<false, GR, RE>), dim3(nblk), dim3(DNW * 64), 0, st, lam, 1, g,             \
                       (const float *)nullptr, K, x, 1, B, T, M, ntile, nq, ticket, aggw, incw, lam_out, HP, PP)
        if (grads && g_real) LBA(true, true, h, part);
        else if (grads) LBA(true, false, h, part);
        else if (g_real) LBA(false, true, (const float *)nullptr, (float *)nullptr);
        else LBA(false, false, (const float *)nullptr, (float *)nullptr);
#undef LBA
    }
    DEER_LAUNCH_CHECK("k_diag_scan_lb");
    if (grads) {
        KTimer _kt("k_diag_grads_sum", st);
        const int nv = 2 + 2 * K;
        hipLaunchKernelGGL(k_diag_grads_sum1, dim3(ntile * nv * DGS), dim3(256), 0, st, (const float *)part, B, ntile, nq,
                           part2);
        hipLaunchKernelGGL(k_diag_grads_sum2, dim3((nv * ntile * DTC + 63) / 64), dim3(64), 0, st,
                           (const double *)part2, K, M, ntile, dlam, dBc);
        DEER_LAUNCH_CHECK("k_diag_grads_sum");
    }
    return DEER_OK;
}

}  // namespace deer
