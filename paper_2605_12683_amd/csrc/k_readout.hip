// Read-out MLP of the diagonal SSM and its mean-squared loss (the LSSM's observation model;
// linear-SSM appendix), forward and backward in one pass over the states:
//   s_t = Wa Re(h_t) + ca            (H hidden units)
//   y_t = Wb relu(s_t) + cb          (No outputs)
//   L   = sum_{b,t} ||y_t - x_{t+1}||^2 / (B No T)        (0-based rows: target row t + 1)
//   dy_t = 2 (y_t - x_{t+1}) / (B No T),  ds_t = (Wb^T dy_t) * 1[s_t > 0]
//   g_t = dL/dRe h_t = Wa^T ds_t     (the cotangent of the reverse scan)
//   dWa = sum ds_t Re(h_t)^T, dca = sum ds_t, dWb = sum dy_t relu(s_t)^T, dcb = sum dy_t
//
// The three products with Wa are dense [16 rows x 64] x [64 x 128] contractions on the fp32
// matrix cores (v_mfma_f32_16x16x4_f32).  A wave takes 16 consecutive (b, t) rows at a time:
//   GEMM1  S^T = Wa H^T     A = Wa (LDS), B = H^T (LDS tile of Re h)
//   GEMM2  G = dS^T Wa      A = dS straight from the GEMM1 accumulator layout (the k index of
//                           the lane group g is 16n + 4g + r, so no data movement), B = Wa (LDS)
//   GEMM3  dWa^T += H^T dS^T, shared by the eight waves of a block: after every round (each
//          wave one tile) wave w accumulates hidden units 16 w .. 16 w + 15 over the 128 rows
//          of all eight tiles (dS and H through LDS), so a wave keeps 16 accumulator floats per
//          lane instead of the whole 128 x 64 dWa, and two waves fit on every SIMD
// The k ordering of GEMM1 is permuted (k-step (jj, q) uses channel 16 jj + 4 g + q in lane group
// g) so that four k-steps read one 16-byte LDS vector of Wa.
#include "common.h"
#include "launch.h"

namespace deer {

namespace {
constexpr int RH = 128;          // hidden units (padded)
constexpr int RM = 64;           // state channels (padded)
constexpr int RNO = 4;           // outputs (padded)
constexpr int RW = 8;            // waves per block (one per 16 hidden units in GEMM3)
constexpr int WS = RM + 4;       // LDS row stride of Wa (16-byte aligned rows)
constexpr int BS = 17;           // LDS row stride of the [hidden][row] tile
// The H tile sits channel-major in LDS, [channel][row] with a row stride of 20 floats: GEMM1
// reads H[row c][channel 16 jj + 4 g + q] and GEMM3 H[row 4 j + g][channel 16 q + c], and with
// 20 = 4 (mod 16) both patterns put the 64 lanes of a read on 64 distinct banks
constexpr int HTS = 20;
constexpr int RPS = RH * RM + RNO * RH + RH + RNO + 1;   // partial floats per wave
constexpr int RPS_PAD = (RPS + 63) & ~63;
}  // namespace

template <bool GRADS>
__global__ __launch_bounds__(RW * 64) void k_readout(const RoArgs ra, const float *__restrict__ h,
                                                     const float *__restrict__ x, int B, int T, float scale,
                                                     float *__restrict__ gout, uint32_t *__restrict__ masks,
                                                     float *__restrict__ part) {
    __shared__ __align__(16) float wa[RH][WS];
    __shared__ float wb[RNO][RH];
    __shared__ float cas[RH];
    __shared__ float cbs[RNO];
    __shared__ float hti[RW][RM][HTS];
    __shared__ float buf[GRADS ? RW : 1][RH][BS];
    __shared__ float dyv[GRADS ? RW : 1][16][RNO];
    __shared__ float lsw[RW];
    const int M = ra.M, H = ra.H, No = ra.No;
    const int tid = threadIdx.x;
    for (int e = tid; e < RH * RM; e += RW * 64) {
        const int i = e / RM, k = e % RM;
        wa[i][k] = (i < H && k < M) ? ra.Wa[i * M + k] : 0.f;
    }
    for (int e = tid; e < RNO * RH; e += RW * 64) {
        const int o = e / RH, i = e % RH;
        wb[o][i] = (o < No && i < H) ? ra.Wb[o * H + i] : 0.f;
    }
    for (int e = tid; e < RH; e += RW * 64) cas[e] = (e < H && ra.ca) ? ra.ca[e] : 0.f;
    if (tid < RNO) cbs[tid] = (tid < No && ra.cb) ? ra.cb[tid] : 0.f;
    __syncthreads();

    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63, g = lane >> 4, c = lane & 15;
    const long rows = (long)B * T;
    const long ntiles = (rows + 15) / 16;
    const int HW = (H + 31) / 32;

    v4f acc3[4];                    // dWa^T tiles [channel tile q] of hidden tile n = wv
    float dwb[RNO][2], dca[2], dcb[RNO], lsum = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) acc3[q] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int o = 0; o < RNO; ++o) dwb[o][0] = dwb[o][1] = dcb[o] = 0.f;
    dca[0] = dca[1] = 0.f;

    // Re h of a tile (one 512-byte row segment per load at M = 64), loaded one tile ahead
    float hv[16];
    // through a buffer resource that ends at the last row: rows past the end, and lanes past M
    // (lane offset >= 2^31), load 0 without branches (the whole offset is in the VGPR, so the
    // range check covers it)
    const int voh = lane < M ? lane * 8 : (int)0x80000000;
    auto load_tile = [&](long tl) {
        const long rb = tl < ntiles ? tl * 16 : rows;
        const long left = rows - rb;
        const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(h + rb * M * 2), (short)0,
                                                          (int)(left < 16 ? left * M * 8 : 16L * M * 8), 0x00020000);
#pragma unroll
        for (int i = 0; i < 16; ++i) hv[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, voh + i * M * 8, 0, 0));
    };
    // rounds are block-uniform (GEMM3 needs every wave at its barriers); a wave whose tile
    // lies past the end works on zero rows, which contribute nothing
    load_tile((long)blockIdx.x * RW + wv);
    for (long base = (long)blockIdx.x * RW; base < ntiles; base += (long)gridDim.x * RW) {
        const long tile = base + wv;
        const long r0 = tile * 16;
#pragma unroll
        for (int i = 0; i < 16; ++i) hti[wv][lane][i] = hv[i];
        load_tile(tile + (long)gridDim.x * RW);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        // GEMM1: acc1[n][r] at lane (g, c) = S^T[hidden 16n + 4g + r][row c]; the eight
        // accumulators are independent, so consecutive matrix-core ops do not wait on each other
        v4f acc1[8];
#pragma unroll
        for (int n = 0; n < 8; ++n) acc1[n] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            float4 bq;
            bq.x = hti[wv][16 * jj + 4 * g + 0][c];
            bq.y = hti[wv][16 * jj + 4 * g + 1][c];
            bq.z = hti[wv][16 * jj + 4 * g + 2][c];
            bq.w = hti[wv][16 * jj + 4 * g + 3][c];
            float4 aq[8];
#pragma unroll
            for (int n = 0; n < 8; ++n) aq[n] = *reinterpret_cast<const float4 *>(&wa[16 * n + c][16 * jj + 4 * g]);
#pragma unroll
            for (int n = 0; n < 8; ++n) acc1[n] = mfma16x16x4(aq[n].x, bq.x, acc1[n]);
#pragma unroll
            for (int n = 0; n < 8; ++n) acc1[n] = mfma16x16x4(aq[n].y, bq.y, acc1[n]);
#pragma unroll
            for (int n = 0; n < 8; ++n) acc1[n] = mfma16x16x4(aq[n].z, bq.z, acc1[n]);
#pragma unroll
            for (int n = 0; n < 8; ++n) acc1[n] = mfma16x16x4(aq[n].w, bq.w, acc1[n]);
        }
        // bias, ReLU, mask bits (bit 4n + r of the lane's hidden units)
        uint32_t mb = 0u;
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float s = acc1[n][r] + cas[16 * n + 4 * g + r];
                const bool pos = s > 0.f;
                acc1[n][r] = pos ? s : 0.f;
                mb |= (pos ? 1u : 0u) << (4 * n + r);
            }
        const long row = r0 + c;
        const bool rok = row < rows;
        if (masks) {
            // word w holds hidden units 32w .. 32w + 31, i.e. tiles n = 2w, 2w + 1
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t word = 0u;
#pragma unroll
                for (int nn = 0; nn < 2; ++nn)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if ((mb >> (4 * (2 * w + nn) + r)) & 1u) word |= 1u << (16 * nn + 4 * g + r);
                word |= (uint32_t)__shfl_xor((int)word, 16, 64);
                word |= (uint32_t)__shfl_xor((int)word, 32, 64);
                if (g == w && w < HW && rok) masks[row * HW + w] = word;
            }
        }
        // outputs y (partial over the lane's 32 hidden units, then over the 4 lane groups)
        float yp[RNO];
#pragma unroll
        for (int o = 0; o < RNO; ++o) {
            float a = 0.f;
#pragma unroll
            for (int n = 0; n < 8; ++n)
#pragma unroll
                for (int r = 0; r < 4; ++r) a = fmaf(wb[o][16 * n + 4 * g + r], acc1[n][r], a);
            a += __shfl_xor(a, 16, 64);
            a += __shfl_xor(a, 32, 64);
            yp[o] = a;
        }
        float dy[RNO];
        {
            // target row t + 1 of sequence b for row = b T + t: x row index row + b + 1, with
            // b from the tile's first row (one scalar division) and the sequence boundaries
            // inside the tile
            // inside the tile (rows past the end read row 1 of a valid sequence, unused)
            const uint32_t Tu = (uint32_t)T;
            const uint32_t b0 = __builtin_amdgcn_readfirstlane((uint32_t)(r0 < rows ? r0 : 0) / Tu);
            const uint32_t rowu = rok ? (uint32_t)row : b0 * Tu;
            uint32_t bq = b0;
            for (int k = 0; k < 16 && rowu >= (bq + 1) * Tu; ++k) ++bq;
            const float *xt = x + ((size_t)rowu + bq + 1) * No;
#pragma unroll
            for (int o = 0; o < RNO; ++o) {
                const bool ok = rok && o < No;
                const float err = ok ? (yp[o] + cbs[o]) - xt[o] : 0.f;
                dy[o] = scale * err;
                if (g == 0) lsum = fmaf(err, err, lsum);
            }
        }
        if (GRADS) {
            // relu(s) and dy to LDS for dWb, dcb
#pragma unroll
            for (int n = 0; n < 8; ++n)
#pragma unroll
                for (int r = 0; r < 4; ++r) buf[wv][16 * n + 4 * g + r][c] = acc1[n][r];
            if (g == 0) {
#pragma unroll
                for (int o = 0; o < RNO; ++o) dyv[wv][c][o] = dy[o];
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            // lane l owns hidden units 2l, 2l + 1 of dWb, dca
#pragma unroll
            for (int rr = 0; rr < 16; ++rr) {
                const float a0 = buf[wv][2 * lane][rr], a1 = buf[wv][2 * lane + 1][rr];
#pragma unroll
                for (int o = 0; o < RNO; ++o) {
                    const float d = dyv[wv][rr][o];
                    dwb[o][0] = fmaf(d, a0, dwb[o][0]);
                    dwb[o][1] = fmaf(d, a1, dwb[o][1]);
                }
            }
            if (g == 0) {
#pragma unroll
                for (int o = 0; o < RNO; ++o) dcb[o] += dy[o];
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        // ds = (Wb^T dy) * mask, in the GEMM1 accumulator layout
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int hid = 16 * n + 4 * g + r;
                float d = 0.f;
#pragma unroll
                for (int o = 0; o < RNO; ++o) d = fmaf(wb[o][hid], dy[o], d);
                acc1[n][r] = ((mb >> (4 * n + r)) & 1u) ? d : 0.f;
            }
        // GEMM2: acc2[q][r] at lane (g, c) = G[row 4g + r][channel 16q + c]
        v4f acc2[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc2[q] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int hid = 16 * n + 4 * g + r;
#pragma unroll
                for (int q = 0; q < 4; ++q) acc2[q] = mfma16x16x4(acc1[n][r], wa[hid][16 * q + c], acc2[q]);
            }
        {
            // g rows r0 + 4 g + r, channels 16 q + c: stores through a resource that ends at the
            // last row (later rows dropped; the whole offset in the VGPR, so the range check
            // covers it), lanes past M get an offset outside it
            const long left = rows - r0 < 0 ? 0 : (rows - r0 < 16 ? rows - r0 : 16);
            const auto rs = __builtin_amdgcn_make_buffer_rsrc(gout + (r0 < rows ? r0 : 0) * M, (short)0,
                                                              (int)(left * M * 4), 0x00020000);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ch = 16 * q + c;
                const int vo = ch < M ? (4 * g * M + ch) * 4 : (int)0x80000000;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc2[q][r]), rs, vo + r * M * 4, 0, 0);
            }
        }
        if (GRADS) {
            // ds to LDS [hidden][row]; dca; GEMM3 over the block's eight tiles
#pragma unroll
            for (int n = 0; n < 8; ++n)
#pragma unroll
                for (int r = 0; r < 4; ++r) buf[wv][16 * n + 4 * g + r][c] = acc1[n][r];
            lds_barrier();
#pragma unroll
            for (int rr = 0; rr < 16; ++rr) {
                dca[0] += buf[wv][2 * lane][rr];
                dca[1] += buf[wv][2 * lane + 1][rr];
            }
#pragma unroll
            for (int w2 = 0; w2 < RW; ++w2) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float bv = buf[w2][16 * wv + c][4 * j + g];
#pragma unroll
                    for (int q = 0; q < 4; ++q) acc3[q] = mfma16x16x4(hti[w2][16 * q + c][4 * j + g], bv, acc3[q]);
                }
            }
            // the next round overwrites hti and buf: every wave is past its reads
            lds_barrier();
        } else {
            // the next tile overwrites hti: every lane is past its reads
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
    }

    // per-block partials: [dWa (RH x RM) | dWb (RNO x RH) | dca (RH) | dcb (RNO) | sum err^2];
    // every wave writes its hidden rows of dWa, the rest is summed over the block's waves
    float *pb = part + (long)blockIdx.x * RPS_PAD;
#pragma unroll
    for (int o = 0; o < RNO; ++o) {
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) dcb[o] += GRADS ? __shfl_xor(dcb[o], off, 64) : 0.f;
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) lsum += __shfl_xor(lsum, off, 64);
    constexpr int RV = RNO * RH + RH + RNO + 1;
    if (GRADS) {
        static_assert(RW * RV <= RW * RH * BS, "block sums fit in the dS tiles");
        float *red = &buf[0][0][0];
        float *rw = red + wv * RV;
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r) pb[(16 * wv + c) * RM + 16 * q + 4 * g + r] = acc3[q][r];
#pragma unroll
        for (int o = 0; o < RNO; ++o) {
            rw[o * RH + 2 * lane] = dwb[o][0];
            rw[o * RH + 2 * lane + 1] = dwb[o][1];
        }
        rw[RNO * RH + 2 * lane] = dca[0];
        rw[RNO * RH + 2 * lane + 1] = dca[1];
        if (lane < RNO) {
            float v = dcb[0];
#pragma unroll
            for (int o = 1; o < RNO; ++o)
                if (lane == o) v = dcb[o];
            rw[RNO * RH + RH + lane] = v;
        }
        if (lane == 0) rw[RV - 1] = lsum;
        __syncthreads();
        for (int e = tid; e < RV; e += RW * 64) {
            float t = 0.f;
#pragma unroll
            for (int w2 = 0; w2 < RW; ++w2) t += red[w2 * RV + e];
            pb[RH * RM + e] = t;
        }
    } else {
        if (lane == 0) lsw[wv] = lsum;
        __syncthreads();
        if (tid == 0) {
            float t = 0.f;
#pragma unroll
            for (int w2 = 0; w2 < RW; ++w2) t += lsw[w2];
            pb[RPS - 1] = t;
        }
    }
}

// float64 sums of the per-block partials: stage 1 over slices of the blocks, stage 2 over slices
constexpr int RO_SLICES = 256;

__global__ __launch_bounds__(256) void k_readout_sum1(const float *__restrict__ part, int nwaves, int only_loss,
                                                      double *__restrict__ part2) {
    const int sl = blockIdx.x;
    const int w0 = (int)((long)nwaves * sl / RO_SLICES), w1 = (int)((long)nwaves * (sl + 1) / RO_SLICES);
    for (int e = only_loss ? RPS - 1 + (int)threadIdx.x : (int)threadIdx.x; e < RPS; e += 256) {
        double s0 = 0.0, s1 = 0.0;
        int w = w0;
        for (; w + 1 < w1; w += 2) {
            s0 += (double)part[(size_t)w * RPS_PAD + e];
            s1 += (double)part[(size_t)(w + 1) * RPS_PAD + e];
        }
        if (w < w1) s0 += (double)part[(size_t)w * RPS_PAD + e];
        part2[(size_t)sl * RPS + e] = s0 + s1;
    }
}

__global__ __launch_bounds__(256) void k_readout_sum2(const double *__restrict__ part2, RoGrads gr, int M, int H,
                                                      int No, float loss_scale, float *__restrict__ loss) {
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= RPS) return;
    if (!loss && e == RPS - 1) return;
    if (!gr.Wa && !gr.Wb && !gr.ca && !gr.cb && e != RPS - 1) return;
    double s = 0.0;
    for (int sl = 0; sl < RO_SLICES; ++sl) s += part2[(size_t)sl * RPS + e];
    if (e < RH * RM) {
        const int i = e / RM, k = e % RM;
        if (gr.Wa && i < H && k < M) gr.Wa[i * M + k] = (float)s;
    } else if (e < RH * RM + RNO * RH) {
        const int o = (e - RH * RM) / RH, i = (e - RH * RM) % RH;
        if (gr.Wb && o < No && i < H) gr.Wb[o * H + i] = (float)s;
    } else if (e < RH * RM + RNO * RH + RH) {
        const int i = e - RH * RM - RNO * RH;
        if (gr.ca && i < H) gr.ca[i] = (float)s;
    } else if (e < RPS - 1) {
        const int o = e - RH * RM - RNO * RH - RH;
        if (gr.cb && o < No) gr.cb[o] = (float)s;
    } else {
        loss[0] = (float)(s * (double)loss_scale);
    }
}

// persistent grid: as many blocks as are resident at once (one pass over the tiles)
static int readout_grid(long rows) {
    static int resident = 0;
    if (!resident) {
        int dev = 0, cus = 0, per = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, k_readout<true>, RW * 64, 0) != hipSuccess || per < 1)
            per = 1;
        resident = cus * per;
    }
    const long ntiles = (rows + 15) / 16;
    const long want = (ntiles + RW - 1) / RW;
    return (int)(want < resident ? want : resident);
}

size_t readout_ws_bytes(int B, int T) {
    const int grid = readout_grid((long)B * T);
    const size_t p1 = ((size_t)grid * RPS_PAD * sizeof(float) + 255) & ~(size_t)255;
    return p1 + (size_t)RO_SLICES * RPS * sizeof(double);
}

int launch_readout(const RoArgs &ra, int B, int T, const float *h, const float *x, float *g, uint32_t *masks,
                   float *loss, const RoGrads &gr, void *ws, hipStream_t st) {
    const int grid = readout_grid((long)B * T);
    const size_t p1 = ((size_t)grid * RPS_PAD * sizeof(float) + 255) & ~(size_t)255;
    float *part = (float *)ws;
    double *part2 = (double *)((char *)ws + p1);
    const float scale = 2.0f / ((float)B * (float)ra.No * (float)T);
    const bool grads = gr.Wa || gr.ca || gr.Wb || gr.cb;
    {
        KTimer _kt("k_readout", st);
        if (grads)
            hipLaunchKernelGGL(k_readout<true>, dim3(grid), dim3(RW * 64), 0, st, ra, h, x, B, T, scale, g, masks, part);
        else
            hipLaunchKernelGGL(k_readout<false>, dim3(grid), dim3(RW * 64), 0, st, ra, h, x, B, T, scale, g, masks,
                               part);
    }
    DEER_LAUNCH_CHECK("k_readout");
    if (grads || loss) {
        KTimer _kt("k_readout_sum", st);
        hipLaunchKernelGGL(k_readout_sum1, dim3(RO_SLICES), dim3(256), 0, st, (const float *)part, grid,
                           grads ? 0 : 1, part2);
        hipLaunchKernelGGL(k_readout_sum2, dim3((RPS + 255) / 256), dim3(256), 0, st, (const double *)part2, gr, ra.M,
                           ra.H, ra.No, 0.5f * scale, loss);
        DEER_LAUNCH_CHECK("k_readout_sum");
    }
    return DEER_OK;
}

}  // namespace deer
