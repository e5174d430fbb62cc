// C ABI of libdeer: argument validation, workspace carving and the host-side Newton loop
// of GTF-DEER (Alg. GTF-DEER).  All device work is queued on the caller's stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <chrono>
#include <vector>

#include "common.h"
#include "launch.h"

namespace deer {

static thread_local char g_err[512] = "";

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

int hip_fail(hipError_t e, const char *what) {
    set_error("%s failed: %s", what, hipGetErrorString(e));
    return DEER_ERR_HIP;
}

// ---- optional per-kernel timing ------------------------------------------------------------
namespace {
struct TimingState {
    std::mutex mu;
    bool on = false;
    std::vector<hipEvent_t> pool;
    std::map<std::string, std::vector<std::pair<hipEvent_t, hipEvent_t>>> recs;
    std::vector<std::string> order;
};
TimingState &tstate() {
    static TimingState s;
    return s;
}
thread_local std::vector<hipEvent_t> t_open;

hipEvent_t take_event(TimingState &s) {
    if (!s.pool.empty()) {
        hipEvent_t e = s.pool.back();
        s.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}
}  // namespace

static thread_local bool t_no_timing = false;
void timing_suppress(bool on) { t_no_timing = on; }
bool timing_suppressed() { return t_no_timing; }

bool timing_on() {
    if (t_no_timing) return false;
    TimingState &s = tstate();
    std::lock_guard<std::mutex> g(s.mu);
    return s.on;
}

void timing_mark(const char *name, hipStream_t st, bool start) {
    TimingState &s = tstate();
    std::lock_guard<std::mutex> g(s.mu);
    hipEvent_t e = take_event(s);
    if (!e) return;
    (void)hipEventRecord(e, st);
    if (start) {
        t_open.push_back(e);
        return;
    }
    if (t_open.empty()) {
        s.pool.push_back(e);
        return;
    }
    hipEvent_t e0 = t_open.back();
    t_open.pop_back();
    auto it = s.recs.find(name);
    if (it == s.recs.end()) {
        s.order.push_back(name);
        it = s.recs.emplace(name, std::vector<std::pair<hipEvent_t, hipEvent_t>>()).first;
    }
    it->second.emplace_back(e0, e);
}

// ---- small utility kernels -------------------------------------------------------------
// z_s = [x_{s+1}; 0] for every (b, s): one sequence per blockIdx.y, four consecutive elements of
// a sequence per thread (a 16-byte store when M is a multiple of 4)
__global__ void k_fill_teacher(int B, int T, int M, int N, const float *__restrict__ x, float *__restrict__ z) {
    const int b = blockIdx.y;
    const size_t n = (size_t)T * M;
    float *zb = z + (size_t)b * n;
    const float *xb = x + ((size_t)b * (T + 1) + 1) * N;   // row s + 1 of x for row s of z
    const size_t n4 = (n + 3) / 4;
    for (size_t e4 = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e4 < n4; e4 += (size_t)gridDim.x * blockDim.x) {
        const size_t e = 4 * e4;
        float v[4];
        size_t s = e / M;
        int i = (int)(e - s * M);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[k] = (e + k < n && i < N) ? xb[s * N + i] : 0.f;
            if (++i == M) {
                i = 0;
                ++s;
            }
        }
        if ((M & 3) == 0) {
            *reinterpret_cast<float4 *>(zb + e) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k)
                if (e + k < n) zb[e + k] = v[k];
        }
    }
}
__global__ void k_fill_i32(int *p, int n, int v) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e < n) p[e] = v;
}
// the iterate of sequence b ended in the second buffer when sel[b] is set: copy it back
__global__ void k_copy_sel(float *__restrict__ z, const float *__restrict__ zalt, const int *__restrict__ sel,
                           size_t seq_elems) {
    const int b = blockIdx.y;
    if (!sel[b]) return;
    float *d = z + (size_t)b * seq_elems;
    const float *s = zalt + (size_t)b * seq_elems;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    if ((seq_elems & 3) == 0 && ((uintptr_t)d & 15) == 0 && ((uintptr_t)s & 15) == 0) {
        const size_t n4 = seq_elems >> 2;
        for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n4; e += stride)
            reinterpret_cast<float4 *>(d)[e] = reinterpret_cast<const float4 *>(s)[e];
    } else {
        for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < seq_elems; e += stride) d[e] = s[e];
    }
}

__global__ void k_fill_f32(float *p, size_t n, float v) {
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n; e += (size_t)gridDim.x * blockDim.x) p[e] = v;
}

int launch_fill_teacher(int B, int T, int M, int N, const float *x, float *z, hipStream_t st) {
    const size_t n4 = ((size_t)T * M + 3) / 4;
    const size_t want = (n4 + 255) / 256;
    const int gx = (int)(want < 1024 ? want : 1024);
    hipLaunchKernelGGL(k_fill_teacher, dim3(gx, B), dim3(256), 0, st, B, T, M, N, x, z);
    DEER_LAUNCH_CHECK("k_fill_teacher");
    return DEER_OK;
}
int launch_fill_i32(int *p, int n, int v, hipStream_t st) {
    hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
    DEER_LAUNCH_CHECK("k_fill_i32");
    return DEER_OK;
}
int launch_fill_f32(float *p, size_t n, float v, hipStream_t st) {
    const int grid = (int)((n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid), dim3(256), 0, st, p, n, v);
    DEER_LAUNCH_CHECK("k_fill_f32");
    return DEER_OK;
}

// ---- workspace carving ---------------------------------------------------------------------
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base((char *)b) {}
    template <class Tp>
    Tp *take(size_t count) {
        Tp *p = base ? (Tp *)(base + off) : nullptr;
        off += (count * sizeof(Tp) + 255) & ~(size_t)255;
        return p;
    }
};

static int chunk_override() {
    const char *e = getenv("DEER_CHUNK");
    return e ? atoi(e) : 0;
}

// DEER_GROUP_MAPS=1 / 0 forces the M <= 16 group maps on (where 32 divides the chunk count) or
// off, whatever the chain count (a tuning and test override)
static int group_maps_override() {
    const char *e = getenv("DEER_GROUP_MAPS");
    return e ? atoi(e) : -1;
}

// DEER_SMALL=0 keeps small fixed-update solves and small adjoints on the general path (a test
// override)
static bool small_path_enabled() {
    const char *e = getenv("DEER_SMALL");
    return !e || atoi(e) != 0;
}

// DEER_PASS_FUSION=0 keeps the M <= 16 fix-up and forward pass in separate kernels where the
// fused pass kernel would apply (a test override)
static bool pass_fusion_allowed() {
    const char *e = getenv("DEER_PASS_FUSION");
    return !e || atoi(e) != 0;
}

// DEER_QUASI_FUSED=0 keeps the vanilla quasi-DEER passes of the adaptive loop in separate
// kernels (a test override)
static bool quasi_fusion_allowed() {
    const char *e = getenv("DEER_QUASI_FUSED");
    return !e || atoi(e) != 0;
}

// Chunk length of the dense scans: enough chains to fill the machine (about 2048 waves),
// and a bounded number of chunks per sequence so that the two-level carry pass stays short
// (1024 for MP <= 32, 512 for MP = 64, whose group pass composes 64 x 64 maps).
// sh_fused: the shallow update without a stored Jacobian, whose fix-up runs 16 chains per block
// (8192 chains keep two of its waves on every SIMD)
static int choose_chunk(int B, int T, int MP, bool sh_fused = false) {
    const int ov = chunk_override();
    if (ov > 0) return ov < T ? ov : T;
    const long total = (long)B * T;
    // MP = 64 runs one chain per wave at two waves per SIMD: 8192 chains keep the tail of a
    // pass (fewer active sequences) spread over the machine
    if (MP == 128) {
        // one 4-wave workgroup per chain, one chain per CU (its staged tiles fill the LDS): about
        // 256 chains, at least 8 steps per chunk (a step is a 128 x 128 x 128 product: on short
        // sequences more chains pay for the longer carry pass)
        long C = (total + 255) / 256;
        if (C < 8) C = 8;
        if (C > T) C = T;
        return (int)C;
    }
    const long target_chains = (MP == 64 || sh_fused) ? 8192L : 2048L * (64 / MP);
    long C = (total + target_chains - 1) / target_chains;
    // at least 16 steps per chunk (8 on the shallow path without a stored Jacobian, whose chunk
    // steps are long chains of dependent products: for short sequences a chunk's serial walk,
    // not the carry pass, sets a pass's time)
    const long minStep = sh_fused ? 8 : 16;
    if (C < minStep) C = minStep;
    const long maxc = MP <= 32 ? 1024 : 512;
    const long minC = (T + maxc - 1) / maxc;
    if (C < minC) C = minC;
    // vanilla M <= 16: whole 16-step tiles (the register-tiled kernels run a partial tile step by
    // step)
    if (MP == 16 && !sh_fused) C = (C + 15) / 16 * 16;
    if (C > T) C = T;
    return (int)C;
}

// Per-sequence control block of the Newton loop (device, 8B words; one device-to-host copy of
// the first 7B reads the results): act | gamma | sel | om | it | norm | status | pv (see
// NewtonDev), then 2B words of max bits for the fixed-iteration mode, the per-chain maxima of
// a pass, and the second iterate buffer.
struct NewtonCtl {
    NewtonDev nd;
    uint32_t *blk;          // start of the 8B-word block
    uint32_t *pv;           // its last B words (NewtonDev::pv of the fused passes)
    uint32_t *norm_bits;
    uint32_t *chain_bits;   // per-chain maxima [2][B * ncs] before the per-sequence reduction
    float *zalt;            // second iterate buffer [B,T,M]
    uint32_t *seq;          // kSeqWords per sequence: the fix-up's fused pass-end control
    bool fused;             // the update takes the pass-end control itself (no k_seq_ctl)
    int lead;               // kernels queued before the first update completes (fused passes: 1)
};

static NewtonCtl carve_ctl(Carver &c, int B, size_t seq_elems, size_t nchains) {
    NewtonCtl n{};
    uint32_t *blk = c.take<uint32_t>(8 * (size_t)B);
    n.blk = blk;
    if (blk) {
        n.pv = blk + 7 * (size_t)B;
        n.nd.act = (int *)blk;
        n.nd.gamma = (float *)(blk + B);
        n.nd.sel = (int *)(blk + 2 * B);
        n.nd.om = (float *)(blk + 3 * B);
        n.nd.it = (int *)(blk + 4 * B);
        n.nd.norm = (float *)(blk + 5 * B);
        n.nd.status = (int *)(blk + 6 * B);
    }
    n.norm_bits = c.take<uint32_t>(2 * (size_t)B);
    n.chain_bits = c.take<uint32_t>(2 * nchains);
    n.zalt = c.take<float>((size_t)B * seq_elems);
    n.seq = c.take<uint32_t>((size_t)kSeqWords * B);
    return n;
}

struct PlrnnWs {
    float *r;
    uint32_t *masks;
    float *P, *v, *carry, *gws;
    float *gmap;   // M <= 16, 32 | chunks: group maps [B][chunks / 32][16 x 16 + 16]
    float *P2, *v2, *gmap2;   // the second set of aggregates of the fused passes (else null)
    NewtonCtl ctl;
    float *gpart;
    double *gpart2;
    int C, ncs, MP;
};

static PlrnnWs carve_plrnn(void *ws, int B, int T, int M, int op, size_t *bytes) {
    PlrnnWs w{};
    w.MP = padded_dim(M);
    w.C = choose_chunk(B, T, w.MP);
    w.ncs = (T + w.C - 1) / w.C;
    const size_t nch = (size_t)B * w.ncs;
    const int MW = (M + 31) / 32;
    Carver c(ws);
    w.masks = c.take<uint32_t>((size_t)B * T * MW);
    w.P = c.take<float>(nch * w.MP * w.MP);
    w.v = c.take<float>(nch * w.MP);
    w.carry = c.take<float>(nch * w.MP);
    w.gws = c.take<float>(carry_ws_floats(w.MP, B, w.ncs));
    // group maps once there are at least 64 blocks of 32 chunks (fewer leave the machine idle
    // while a block composes its maps; the carry kernel is then cheaper)
    const int gov = group_maps_override();
    const bool gm = w.MP == 16 && w.ncs % 32 == 0 && (gov < 0 ? nch >= 2048 : gov > 0);
    w.gmap = gm ? c.take<float>((size_t)B * (w.ncs / 32) * 272) : nullptr;
    // fused passes: group maps, whole chunks of whole tiles
    if (op == DEER_OP_SOLVE && gm && (long)w.C * w.ncs == T && w.C % 16 == 0 && pass_fusion_allowed()) {
        w.P2 = c.take<float>(nch * 256);
        w.v2 = c.take<float>(nch * 16);
        w.gmap2 = c.take<float>((size_t)B * (w.ncs / 32) * 272);
    }
    if (op == DEER_OP_SOLVE) {
        w.ctl = carve_ctl(c, B, (size_t)T * M, nch);
        w.r = c.take<float>((size_t)B * T * M);
    } else {
        w.gpart = c.take<float>(nch * w.MP * (w.MP + 2));
        w.gpart2 = c.take<double>(reduce_gpart_ws_bytes(w.MP) / sizeof(double));
    }
    *bytes = c.off;
    return w;
}

struct DenseWs {
    float *P, *v, *carry, *gws;
    int C, ncs, MP;
};

static DenseWs carve_dense(void *ws, int B, int T, int M, size_t *bytes, bool sh_fused = false) {
    DenseWs w{};
    w.MP = padded_dim(M);
    w.C = choose_chunk(B, T, w.MP, sh_fused);
    w.ncs = (T + w.C - 1) / w.C;
    const size_t nch = (size_t)B * w.ncs;
    Carver c(ws);
    w.P = c.take<float>(nch * w.MP * w.MP);
    w.v = c.take<float>(nch * w.MP);
    w.carry = c.take<float>(nch * w.MP);
    w.gws = c.take<float>(carry_ws_floats(w.MP, B, w.ncs));
    *bytes = c.off;
    return w;
}

struct ShWs {
    float *r, *J, *g, *lam, *part;
    uint32_t *masks;
    DenseWs d;
    NewtonCtl ctl;
};

// The shallow solve and adjoint without a stored Jacobian (the forced Jacobians rebuilt from the
// hidden masks by the chunk products and applied as Jacobian-vector products in the fix-ups); on
// unless DEER_SH_FUSED=0, for the identity read-out at M <= 64 within the kernels' tile limits.
static bool sh_fused(int M, int L) {
    const char *e = getenv("DEER_SH_FUSED");
    if (e && atoi(e) == 0) return false;
    return shfused_supported(M, L);
}

// Newton passes of the fused shallow path: residual and masks on the matrix cores (the pass's
// own masks; the fixed-order float32 decision of k_resjac_shplrnn is kept for the masks a
// caller receives and for the adjoint); on unless DEER_SH_RESMFMA=0
static bool sh_res_mfma() {
    const char *e = getenv("DEER_SH_RESMFMA");
    return !e || atoi(e) != 0;
}

static ShWs carve_sh(void *ws, int B, int T, int M, int L, int op, bool need_g, bool need_lam, size_t *bytes,
                     bool stored_J = true) {
    ShWs w{};
    const int LW = (L + 31) / 32;
    Carver c(ws);
    w.masks = c.take<uint32_t>((size_t)B * T * LW);
    w.J = stored_J ? c.take<float>((size_t)B * T * M * M) : nullptr;
    if (op == DEER_OP_SOLVE) {
        const int C = choose_chunk(B, T, padded_dim(M), !stored_J);
        w.ctl = carve_ctl(c, B, (size_t)T * M, (size_t)B * ((T + C - 1) / C));
        w.r = c.take<float>((size_t)B * T * M);
    } else {
        if (need_g) w.g = c.take<float>((size_t)B * T * M);
        if (need_lam) w.lam = c.take<float>((size_t)B * T * M);
        int nb = 0;
        w.part = c.take<float>(sh_grads_part_floats(M, L, &nb));
    }
    size_t dbytes = 0;
    w.d = carve_dense(ws ? (char *)ws + c.off : nullptr, B, T, M, &dbytes, !stored_J);
    *bytes = c.off + dbytes;
    return w;
}

// quasi-DEER workspace: right-hand side and coefficients [B,T,M], chunk aggregates and
// carries [chains, MP]; solve: the Newton control block and second iterate; adjoint: the
// per-chain gradient partials and their float64 slices
// (shallow PLRNN, L > 0: the hidden-unit masks; adjoint: the adjoint itself when the caller
// does not keep it, and the partial sums of the shallow gradient kernel)
struct QuasiWs {
    float *rhs, *coef, *P, *v, *carry;
    float *P2, *v2;      // vanilla solve: the second set of chunk aggregates of the fused passes
    double *gm, *gm2;    // and the two sets of group maps [B][chunks / group][2][MP]
    NewtonCtl ctl;
    float *gpart;
    double *gpart2;
    uint32_t *masks;
    float *lam, *part;
    int C, ncs, MP;
};

// The vanilla solve is carved for the fused passes (chunk count per sequence padded to a whole
// number of the pass kernel's groups; the separate kernels take the empty padding chunks too).
static QuasiWs carve_quasi(void *ws, int B, int T, int M, int L, int op, size_t *bytes) {
    QuasiWs w{};
    w.MP = padded_dim(M);
    w.C = qdeer_chunk_len(B, T, M);
    w.ncs = (T + w.C - 1) / w.C;
    const bool fused = op == DEER_OP_SOLVE && L == 0;
    const int GS = fused ? qdeer_pass_group(M) : 1;
    if (fused)
        while (w.ncs > qdeer_pass_max_chunks(M)) {
            w.C *= 2;
            w.ncs = (T + w.C - 1) / w.C;
        }
    w.ncs = (w.ncs + GS - 1) / GS * GS;
    const size_t nch = (size_t)B * w.ncs;
    Carver c(ws);
    w.coef = c.take<float>((size_t)B * T * M);
    w.P = c.take<float>(nch * w.MP);
    w.v = c.take<float>(nch * w.MP);
    w.carry = c.take<float>(nch * w.MP);
    if (L > 0) w.masks = c.take<uint32_t>((size_t)B * T * ((L + 31) / 32));
    if (op == DEER_OP_SOLVE) {
        w.rhs = c.take<float>((size_t)B * T * M);
        w.ctl = carve_ctl(c, B, (size_t)T * M, nch);
        if (fused) {
            const size_t ngm = (size_t)B * (w.ncs / GS) * 2 * w.MP;
            w.P2 = c.take<float>(nch * w.MP);
            w.v2 = c.take<float>(nch * w.MP);
            w.gm = c.take<double>(ngm);
            w.gm2 = c.take<double>(ngm);
        }
    } else if (L > 0) {
        w.lam = c.take<float>((size_t)B * T * M);
        int nb = 0;
        w.part = c.take<float>(sh_grads_part_floats(M, L, &nb));
    } else {
        w.gpart = c.take<float>(nch * w.MP * (w.MP + 2));
        w.gpart2 = c.take<double>(reduce_gpart_ws_bytes(w.MP) / sizeof(double));
    }
    *bytes = c.off;
    return w;
}

static int quasi_L(const deer_model *m) { return m->kind == DEER_SHPLRNN ? m->L : 0; }

static int check_shallow_limits(const deer_model *m) {
    const size_t cap = 64 * 1024;
    if (m->M > 64) {   // width-128 kernels: W1 and W2 in LDS
        if (big_resjac_lds(m->M, m->L) > cap || big_jacform_lds(m->L) > cap || big_grads_lds(m->M, m->L) > cap) {
            set_error("shallow PLRNN with M=%d, L=%d exceeds the 64 KiB LDS tiles of the width-128 kernels "
                      "(M > 64 needs L <= 62 and M L <= 7936)", m->M, m->L);
            return DEER_ERR_INVALID_ARG;
        }
        return DEER_OK;
    }
    if (sh_resjac_lds(m->M, m->L) > cap || sh_jacform_lds(m->M, m->L) > cap) {
        set_error("shallow PLRNN with M=%d, L=%d exceeds the 64 KiB LDS tiles of this build (need M*L <= 8192 "
                  "for M <= 32)", m->M, m->L);
        return DEER_ERR_INVALID_ARG;
    }
    return DEER_OK;
}



static int check_common(const deer_model *m, const deer_forcing *f, int B, int T) {
    if (!m || !f) { set_error("model/forcing pointer is NULL"); return DEER_ERR_INVALID_ARG; }
    if (B <= 0 || T <= 0) { set_error("B and T must be positive (B=%d, T=%d)", B, T); return DEER_ERR_INVALID_ARG; }
    if (!(f->alpha >= 0.0f && f->alpha <= 1.0f)) { set_error("alpha must lie in [0, 1]"); return DEER_ERR_INVALID_ARG; }
    if (m->M <= 0) { set_error("M must be positive"); return DEER_ERR_INVALID_ARG; }
    if (m->kind == DEER_PLRNN || m->kind == DEER_SHPLRNN) {
        const int mmax = m->kind == DEER_SHPLRNN && !f->obs ? 128 : 64;
        if (m->M > mmax) {
            set_error("M=%d unsupported (dense scans support M <= %d for this model and forcing)", m->M, mmax);
            return DEER_ERR_INVALID_ARG;
        }
        if (f->obs) {
            if (f->n_forced < 1 || f->n_forced > 64) {
                set_error("with an observation matrix, n_forced (its row count) must lie in [1, 64]");
                return DEER_ERR_INVALID_ARG;
            }
        } else if (f->n_forced < 0 || f->n_forced > m->M) {
            set_error("n_forced must lie in [0, M]");
            return DEER_ERR_INVALID_ARG;
        }
        if (!m->A || !m->W) { set_error("model parameters A and W are required"); return DEER_ERR_INVALID_ARG; }
        if (m->kind == DEER_SHPLRNN) {
            if (m->L <= 0 || m->L > 1024 || !m->W2) { set_error("shallow PLRNN needs W2 and 1 <= L <= 1024"); return DEER_ERR_INVALID_ARG; }
        }
    } else if (m->kind == DEER_DIAG_SSM) {
        if (!m->A || !m->W) { set_error("DIAG_SSM needs lambda (A) and Bc (W)"); return DEER_ERR_INVALID_ARG; }
        if (m->L <= 0 || m->L > 4) { set_error("DIAG_SSM input dimension L must lie in [1, 4]"); return DEER_ERR_INVALID_ARG; }
    } else {
        set_error("unknown model kind %d", m->kind);
        return DEER_ERR_INVALID_ARG;
    }
    if ((long)B * (long)T > (1L << 31) / 1) { set_error("B*T too large"); return DEER_ERR_INVALID_ARG; }
    if (f->T_w < 0 || (f->T_w > 0 && f->T_w >= T)) {
        set_error("T_w must satisfy 0 <= T_w < T (T_w=%d, T=%d)", f->T_w, T);
        return DEER_ERR_INVALID_ARG;
    }
    if (f->T_w > 0 && m->kind == DEER_DIAG_SSM) {
        set_error("the latent warm-up applies to the PLRNN kinds");
        return DEER_ERR_INVALID_ARG;
    }
    if (f->obs && m->kind == DEER_DIAG_SSM) {
        set_error("an observation matrix applies to the PLRNN kinds");
        return DEER_ERR_INVALID_ARG;
    }
    return DEER_OK;
}

// entry points that take the identity read-out only
static int no_obs(const deer_forcing *f, const char *entry) {
    if (f && f->obs) {
        set_error("%s: a general observation matrix is supported by deer_solve and deer_adjoint only", entry);
        return DEER_ERR_INVALID_ARG;
    }
    return DEER_OK;
}

static int check_quasi(const deer_model *m, const deer_forcing *f, int B, int T) {
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if ((rc = no_obs(f, "quasi-DEER"))) return rc;
    if (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN) {
        set_error("quasi-DEER is built for the PLRNN kinds only");
        return DEER_ERR_INVALID_ARG;
    }
    if (m->M > 64) {
        set_error("quasi-DEER supports M <= 64");
        return DEER_ERR_INVALID_ARG;
    }
    if (m->kind == DEER_SHPLRNN) return check_shallow_limits(m);
    return DEER_OK;
}

static int check_ws(void *ws, size_t have, size_t need) {
    if (need == 0) return DEER_OK;
    if (!ws || have < need) {
        set_error("workspace too small: need %zu bytes, have %zu", need, ws ? have : (size_t)0);
        return DEER_ERR_WORKSPACE;
    }
    if (((uintptr_t)ws & 255u) != 0) { set_error("workspace must be 256-byte aligned"); return DEER_ERR_WORKSPACE; }
    return DEER_OK;
}

static size_t diag_bytes(int B, int T, int M, int K, int op) {
    return op == DEER_OP_ADJOINT ? diag_adjoint_ws_bytes(B, T, M, K) : diag_scan_ws_bytes(B, T, M);
}

// Newton loop shared by the PLRNN kinds.  `update(act, gamma, zsel, z, zalt, mark, pass_no)`
// queues one Newton update of the sequences whose device flag is set (all, when act is null),
// linearised with the per-sequence factor gamma (gamma J~; null: 1), reading each sequence's
// iterate from the buffer zsel selects and writing iterate + Delta to the other one (zsel
// null and zalt == z: in place), and leaves per-chain max|Delta| and max|z| bits in
// ctl.chain_bits; with a mark, the pass writes pass_no to it as it starts.
//
// With a convergence test (fixed_iters == 0) the test and the update safeguard run on the
// device after every pass (in the fix-up, or k_seq_ctl): an update that is not finite, or
// whose max|Delta| exceeds step_bound (1 + max|z|), is not kept and the sequence is retried
// with gamma < 1; gamma returns to 1 over accepted updates.  gamma = 1 is the exact Newton
// step, gamma = 0 the fixed-point step z_t <- F(z~_{t-1}); every gamma keeps the fixed point
// and the prefix property.  A sequence that stops clears its flag on the device and in a
// pinned host block that also receives its results, so the host follows the device without
// copies; a sequence frozen while passes are queued makes them skip it, and once every
// sequence is frozen the passes still queued skip everything.  The call returns when every
// sequence has stopped (or at the iteration cap); z is then complete in stream order.
constexpr float kDefaultStepBound = 1e3f;
constexpr NewtonDamp kDamp = {1.f / 64, 4.f, 4.f, 1e-4f};
constexpr int kFirstBatch = 4, kBatch = 1;

// Pinned, device-coherent host block of the Newton loop, one per host thread, reserved by
// deer_host_reserve (the solves allocate nothing): act | it | norm | status (cap words each; see
// NewtonDev), then the pass mark.  Passes are numbered per thread; the M <= 16 forward pass
// writes its number to the mark as it starts.
struct HostBlk {
    int *base = nullptr;
    size_t cap = 0;
    uint32_t next_pass = 1;   // number of the next marked pass
};
static thread_local HostBlk t_host;

static int host_reserve(int B) {
    if ((size_t)B <= t_host.cap) return DEER_OK;
    if (t_host.base) (void)hipHostFree(t_host.base);
    t_host.base = nullptr;
    t_host.cap = 0;
    DEER_HIP(hipHostMalloc((void **)&t_host.base, (4 * (size_t)B + 32) * sizeof(int), hipHostMallocCoherent));
    t_host.cap = (size_t)B;
    // no pass of this thread is pending (every earlier solve returned after its last mark)
    *(uint32_t *)(t_host.base + 4 * t_host.cap) = t_host.next_pass - 1;
    return DEER_OK;
}

// A solve with a tolerance needs the calling thread's block to hold B sequences; checked before
// any device work is queued.
static int check_host_reserved(int B) {
    if ((size_t)B <= t_host.cap) return DEER_OK;
    set_error("solves with a tolerance report through a pinned host block of the calling thread: it holds %zu "
              "sequences, %d are needed (call deer_host_reserve(%d) on this thread first)",
              t_host.cap, B, B);
    return DEER_ERR_INVALID_ARG;
}

static int host_block(int B, NewtonDev &nd, uint32_t **mark) {
    int rc = check_host_reserved(B);
    if (rc) return rc;
    int *p = t_host.base;
    const size_t cap = t_host.cap;
    nd.hact = p;
    nd.hit = p + cap;
    nd.hnorm = (float *)(p + 2 * cap);
    nd.hstat = p + 3 * cap;
    *mark = (uint32_t *)(p + 4 * cap);
    return DEER_OK;
}

// Waits until the pass mark has reached `want` (in wrapping order).  The stream is queried only
// after a long wait (a runtime call while the device works delays the following kernels), so
// that a stream that ran dry without the mark is an error, not a hang.
static int wait_mark(const uint32_t *mark, uint32_t want, hipStream_t st) {
    auto reached = [&]() { return (int32_t)(__atomic_load_n(mark, __ATOMIC_ACQUIRE) - want) >= 0; };
    using clk = std::chrono::steady_clock;
    const auto t0 = clk::now();
    for (unsigned spin = 1;; ++spin) {
        if (reached()) return DEER_OK;
        if ((spin & 4095u) == 0u && clk::now() - t0 > std::chrono::milliseconds(200)) {
            const hipError_t e = hipStreamQuery(st);
            if (e == hipSuccess) {
                if (reached()) return DEER_OK;
                set_error("the stream finished without the forward pass's mark");
                return DEER_ERR_HIP;
            }
            if (e != hipErrorNotReady) return hip_fail(e, "hipStreamQuery");
        }
        __builtin_ia32_pause();
    }
}

template <class Update>
static int newton_loop(const deer_solve_opts *o, int B, size_t seq_elems, int ncs, const NewtonCtl &ctl, float *z,
                       Update update, std::vector<int> &it, std::vector<float> &norm, bool &nonfinite,
                       std::vector<int> &act, hipStream_t st) {
    const int fixed = o->fixed_iters > 0 ? o->fixed_iters : 0;
    const int max_iter = o->max_iter > 0 ? o->max_iter : 500;
    const float bound = o->step_bound == 0.f ? kDefaultStepBound : o->step_bound;
    int rc;
    if (fixed) {
        for (int k = 0; k < fixed; ++k)
            if ((rc = update(nullptr, nullptr, nullptr, z, z, nullptr, 0u))) return rc;
        if ((rc = launch_seq_max(ctl.chain_bits, nullptr, ctl.norm_bits, B, ncs, st))) return rc;
        std::vector<uint32_t> nb(B, 0);
        DEER_HIP(hipMemcpyAsync(nb.data(), ctl.norm_bits, B * sizeof(uint32_t), hipMemcpyDeviceToHost, st));
        DEER_HIP(hipStreamSynchronize(st));
        for (int b = 0; b < B; ++b) {
            memcpy(&norm[b], &nb[b], 4);
            it[b] = fixed;
            if (!isfinite(norm[b])) nonfinite = true;
        }
        return DEER_OK;
    }
    NewtonDev nd = ctl.nd;
    uint32_t *mark = nullptr;
    if ((rc = host_block(B, nd, &mark))) return rc;
    int *const hact = nd.hact;
    for (int b = 0; b < B; ++b) hact[b] = 1;   // no kernel of this stream that writes it is pending
    if ((rc = launch_ctl_init(nd, ctl.seq, B, st))) return rc;
    auto all_stopped = [&]() {
        bool any = false;
        for (int b = 0; b < B; ++b) any |= __atomic_load_n(hact + b, __ATOMIC_ACQUIRE) != 0;
        return !any;
    };
    bool stopped = false;
    if (ctl.fused) {
        // Passes whose last kernel takes the pass-end control (the vanilla M <= 16 and shallow
        // fix-ups, the one-kernel passes).  The first kernel of pass p marks its start,
        // when every earlier pass, and so the decisions of pass p - 1, is complete.  The host
        // keeps one pass queued ahead: once pass p has started it reads the flags as of pass
        // p - 1 and queues pass p + 1 (a whole pass of time to do so), so the device does not
        // wait for the host and one pass runs past convergence (it skips every sequence).  The
        // loop ends only after the mark of the last queued pass, so no mark is pending.
        int passes = 0;
        uint32_t last = 0u;   // number of the last pass queued
        auto queue = [&]() {
            const uint32_t no = t_host.next_pass;
            const int r = update(nd.act, nd.gamma, nd.sel, z, ctl.zalt, mark, no);
            if (++t_host.next_pass == 0u) t_host.next_pass = 1u;   // 0 marks "no aggregates"
            last = no;
            ++passes;
            return r;
        };
        const int cap = max_iter + ctl.lead;
        rc = queue();
        if (!rc && passes < cap) rc = queue();
        while (!rc) {
            if ((rc = wait_mark(mark, last, st))) break;
            if ((stopped = all_stopped())) break;
            if (passes >= cap) break;
            rc = queue();
        }
        if (rc) return rc;
    } else {
        // Long passes: batches of passes with an event after each; the host waits for the batch
        // just queued (the wait is small next to a pass, and a pass queued past convergence is
        // not).
        hipEvent_t ev = nullptr;
        DEER_HIP(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
        int passes = 0, batch = kFirstBatch;
        while (passes < max_iter) {
            const int n = batch < max_iter - passes ? batch : max_iter - passes;
            for (int j = 0; j < n && !rc; ++j) {
                rc = update(nd.act, nd.gamma, nd.sel, z, ctl.zalt, nullptr, 0u);
                if (!rc) rc = launch_seq_ctl(ctl.chain_bits, nd, B, ncs, o->tol, bound, kDamp, st);
            }
            if (rc) break;
            hipError_t e = hipEventRecord(ev, st);
            if (e == hipSuccess) e = hipEventSynchronize(ev);
            if (e != hipSuccess) {
                rc = hip_fail(e, "hipEventRecord / hipEventSynchronize");
                break;
            }
            passes += n;
            batch = kBatch;
            if ((stopped = all_stopped())) break;
        }
        (void)hipEventDestroy(ev);
        if (rc) return rc;
    }
    // sequences whose iterate ended in the second buffer are copied back on the device (one
    // launch, no host decision)
    {
        const size_t n4 = (seq_elems + 3) / 4;
        const unsigned gx = (unsigned)((n4 + 255) / 256 < 256 ? (n4 + 255) / 256 : 256);
        hipLaunchKernelGGL(k_copy_sel, dim3(gx, B), dim3(256), 0, st, z, (const float *)ctl.zalt,
                           (const int *)nd.sel, seq_elems);
        DEER_LAUNCH_CHECK("k_copy_sel");
    }
    if (stopped) {
        // every sequence has stopped: its results are in the host block, and the kernels still
        // queued only skip (z is complete in stream order)
        for (int b = 0; b < B; ++b) {
            act[b] = 0;
            it[b] = nd.hit[b];
            norm[b] = nd.hnorm[b];
            if (nd.hstat[b] == 2) nonfinite = true;
        }
        return DEER_OK;
    }
    // iteration cap reached: the control block is read once
    std::vector<uint32_t> h(7 * (size_t)B);
    DEER_HIP(hipMemcpyAsync(h.data(), ctl.blk, h.size() * sizeof(uint32_t), hipMemcpyDeviceToHost, st));
    DEER_HIP(hipStreamSynchronize(st));
    for (int b = 0; b < B; ++b) {
        act[b] = (int)h[b];
        it[b] = (int)h[4 * (size_t)B + b];
        memcpy(&norm[b], &h[5 * (size_t)B + b], 4);
        if (h[6 * (size_t)B + b] == 2u) nonfinite = true;
    }
    return DEER_OK;
}

static int finish_solve(const deer_solve_opts *o, int B, const std::vector<int> &it, const std::vector<float> &norm,
                        bool nonfinite, const std::vector<int> &act, int32_t *iters, float *final_norm) {
    if (iters) for (int b = 0; b < B; ++b) iters[b] = it[b];
    if (final_norm) for (int b = 0; b < B; ++b) final_norm[b] = norm[b];
    if (nonfinite) {
        set_error("a Newton update produced a non-finite value");
        return DEER_ERR_NONFINITE;
    }
    if (o->fixed_iters <= 0) {
        for (int b = 0; b < B; ++b)
            if (act[b]) {
                set_error("sequence %d not converged after %d Newton updates (last max|dz| = %g)", b, it[b], norm[b]);
                return DEER_ERR_NOT_CONVERGED;
            }
    }
    return DEER_OK;
}

static int init_guess(const deer_solve_opts *o, int B, int T, int M, int N, const float *x, float *z, hipStream_t st) {
    if (o->init == DEER_INIT_TEACHER) return launch_fill_teacher(B, T, M, N, x, z, st);
    if (o->init == DEER_INIT_ZERO) return launch_fill_f32(z, (size_t)B * T * M, 0.f, st);
    return DEER_OK;
}

// J~ of every step of the shallow model into J; with a latent warm-up, steps 0..T_w take P_1
// (alpha = 1; step 0's Jacobian only multiplies the fixed initial state's zero update) and the
// rest P_alpha
static int jacform_sh(const ShArgs &a, const uint32_t *masks, float *J, const int *active, const float *gamma,
                      hipStream_t st) {
    if (a.tw <= 0) return launch_jacform_shplrnn(a, masks, J, active, gamma, st);
    ShArgs w = a;
    w.alpha = 1.f;
    w.t_lo = 0;
    w.t_hi = a.tw + 1;
    int rc = launch_jacform_shplrnn(w, masks, J, active, gamma, st);
    if (rc || a.tw + 1 >= a.T) return rc;
    w.alpha = a.alpha;
    w.t_lo = a.tw + 1;
    w.t_hi = a.T;
    return launch_jacform_shplrnn(w, masks, J, active, gamma, st);
}

static int solve_plrnn(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T,
                       const float *x, const float *z0, float *z, uint32_t *masks, int32_t *iters, float *final_norm,
                       void *ws, size_t ws_bytes, hipStream_t st) {
    size_t need = 0;
    carve_plrnn(nullptr, B, T, m->M, DEER_OP_SOLVE, &need);
    int rc = check_ws(ws, ws_bytes, need);
    if (rc) return rc;
    PlrnnWs w = carve_plrnn(ws, B, T, m->M, DEER_OP_SOLVE, &need);
    PlrnnArgs a{m->A, m->W, m->h, f->alpha, f->n_forced, x, z0, B, T, m->M};
    a.tw = f->T_w;
    if ((rc = init_guess(o, B, T, m->M, f->n_forced, x, z, st))) return rc;
    std::vector<int> act(B, 1), it(B, 0);
    std::vector<float> norm(B, NAN);
    bool nonfinite = false;
    if (a.tw == 0 && small_path_enabled() && newton_small_fits(m->M, T, o->fixed_iters)) {
        // every update in one launch; the last update's norms read once
        if ((rc = launch_newton_small(a, z, o->fixed_iters, w.ctl.norm_bits, st))) return rc;
        std::vector<uint32_t> nb(B, 0);
        DEER_HIP(hipMemcpyAsync(nb.data(), w.ctl.norm_bits, B * sizeof(uint32_t), hipMemcpyDeviceToHost, st));
        DEER_HIP(hipStreamSynchronize(st));
        for (int b = 0; b < B; ++b) {
            memcpy(&norm[b], &nb[b], 4);
            it[b] = o->fixed_iters;
            if (!isfinite(norm[b])) nonfinite = true;
        }
        if (masks && (rc = launch_resjac_plrnn(a, z, nullptr, nullptr, nullptr, masks, nullptr, st))) return rc;
        return finish_solve(o, B, it, norm, nonfinite, act, iters, final_norm);
    }
    // M <= 16: the fix-up also takes the pass-end control of the adaptive loop
    NewtonCtl ctl = w.ctl;
    ctl.fused = w.MP == 16 && o->fixed_iters <= 0;
    // one kernel per pass: the fix-up of the previous update and the forward pass of the next
    const bool pass16 = ctl.fused && w.P2;
    if (pass16) {
        ctl.nd.pv = ctl.pv;
        ctl.lead = 1;
    }
    uint32_t *mark_unused = nullptr;
    if (ctl.fused && (rc = host_block(B, ctl.nd, &mark_unused))) return rc;
    const FusedCtl fc{ctl.nd, ctl.seq, o->tol, o->step_bound == 0.f ? kDefaultStepBound : o->step_bound, kDamp};
    auto update = [&](const int *dact, const float *gam, const int *zsel, float *zb, float *za, uint32_t *mark,
                      uint32_t pass_no) -> int {
        int r;
        if (pass16) {   // aggregates alternate between the two sets
            const bool odd = pass_no & 1u;
            return launch_newton_pass16(a, zb, za, odd ? w.P2 : w.P, odd ? w.v2 : w.v, odd ? w.gmap2 : w.gmap,
                                        odd ? w.P : w.P2, odd ? w.v : w.v2, odd ? w.gmap : w.gmap2, w.C, w.ncs, fc,
                                        mark, pass_no, st);
        }
        // M <= 16: each wave's four chunks are composed in the forward pass, one kernel walks
        // the composed maps, and the fix-up applies the per-chunk prefix maps
        // 32 | chunks: the forward pass also composes each block's eight wave maps into a
        // group map and the fix-up walks the group maps itself (no carry kernel)
        const bool wm = w.MP == 16 && w.ncs % 4 == 0, gm = w.gmap != nullptr;
        const int mode = gm ? 2 : (wm ? 1 : 0);
        if ((r = launch_newton_product_plrnn(a, zb, za, zsel, w.r, w.masks, w.P, w.v, dact, gam, w.C, w.ncs, mode,
                                             w.gmap, mark, pass_no, st)))
            return r;
        if (gm) r = 0;
        else if (wm) r = launch_carry_walk16(false, w.P, w.v, w.carry, dact, B, w.ncs, st);
        else r = launch_carry(w.MP, false, w.P, w.v, w.carry, dact, nullptr, B, w.ncs, w.gws, st);
        if (r) return r;
        return launch_fixup_fwd_plrnn(a, w.masks, w.r, w.carry, zb, za, zsel, w.ctl.chain_bits, dact, gam, w.C, w.ncs,
                                      wm ? w.P : nullptr, wm ? w.v : nullptr, w.gmap,
                                      (ctl.fused && dact) ? &fc : nullptr, st);
    };
    if ((rc = newton_loop(o, B, (size_t)T * m->M, w.ncs, ctl, z, update, it, norm, nonfinite, act, st))) return rc;
    if (masks) {
        if ((rc = launch_resjac_plrnn(a, z, nullptr, nullptr, nullptr, masks, nullptr, st))) return rc;
    }
    return finish_solve(o, B, it, norm, nonfinite, act, iters, final_norm);
}

static int solve_shplrnn(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T,
                         const float *x, const float *z0, float *z, uint32_t *masks, int32_t *iters,
                         float *final_norm, void *ws, size_t ws_bytes, hipStream_t st) {
    int rc = check_shallow_limits(m);
    if (rc) return rc;
    const bool fused = sh_fused(m->M, m->L);
    size_t need = 0;
    carve_sh(nullptr, B, T, m->M, m->L, DEER_OP_SOLVE, false, false, &need, !fused);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    ShWs w = carve_sh(ws, B, T, m->M, m->L, DEER_OP_SOLVE, false, false, &need, !fused);
    ShArgs a{m->A, m->W, m->W2, m->h, m->h2, f->alpha, f->n_forced, x, z0, B, T, m->M, m->L};
    a.tw = f->T_w;
    if ((rc = init_guess(o, B, T, m->M, f->n_forced, x, z, st))) return rc;
    std::vector<int> act(B, 1), it(B, 0);
    std::vector<float> norm(B, NAN);
    bool nonfinite = false;
    const DenseWs &d = w.d;
    // adaptive loop on the path without a stored Jacobian: the fix-up takes the pass-end control
    // and the residual kernel marks each pass's start, so passes are queued one ahead with no
    // control kernel and no host wait per pass
    NewtonCtl ctl = w.ctl;
    ctl.fused = fused && sh_res_mfma() && o->fixed_iters <= 0;
    if (ctl.fused) {
        uint32_t *mark_unused = nullptr;
        if ((rc = host_block(B, ctl.nd, &mark_unused))) return rc;
    }
    const FusedCtl fc{ctl.nd, ctl.seq, o->tol, o->step_bound == 0.f ? kDefaultStepBound : o->step_bound, kDamp};
    auto update = [&](const int *dact, const float *gam, const int *zsel, float *zb, float *za, uint32_t *mark,
                      uint32_t pass_no) -> int {
        int r;
        if (fused && sh_res_mfma()) {
            if ((r = launch_resjac_shmfma(a, zb, za, zsel, w.r, w.masks, dact, st, mark, pass_no))) return r;
        } else if ((r = launch_resjac_shplrnn(a, zb, za, zsel, nullptr, w.r, w.masks, dact, st))) {
            return r;
        }
        if (fused) {
            if ((r = launch_chunk_product_shfused(false, a, w.masks, w.r, -1.f, gam, d.P, d.v, dact, d.C, d.ncs, st)))
                return r;
            if ((r = launch_carry(d.MP, false, d.P, d.v, d.carry, dact, nullptr, B, d.ncs, d.gws, st))) return r;
            return launch_fixup_shjvp(false, a, w.masks, w.r, -1.f, gam, d.carry, zb, za, zsel, w.ctl.chain_bits, dact,
                                      d.C, d.ncs, st, (ctl.fused && dact) ? &fc : nullptr);
        }
        if ((r = jacform_sh(a, w.masks, w.J, dact, gam, st))) return r;
        if ((r = launch_chunk_product_dense(false, B, T, m->M, w.J, w.r, -1.f, d.P, d.v, dact, d.C, d.ncs, st))) return r;
        if ((r = launch_carry(d.MP, false, d.P, d.v, d.carry, dact, nullptr, B, d.ncs, d.gws, st))) return r;
        return launch_fixup_dense(0, B, T, m->M, w.J, w.r, -1.f, d.carry, zb, za, zsel, w.ctl.chain_bits, dact, d.C,
                                  d.ncs, st);
    };
    if ((rc = newton_loop(o, B, (size_t)T * m->M, d.ncs, ctl, z, update, it, norm, nonfinite, act, st))) return rc;
    if (masks) {
        if ((rc = launch_resjac_shplrnn(a, z, nullptr, nullptr, nullptr, nullptr, masks, nullptr, st))) return rc;
    }
    return finish_solve(o, B, it, norm, nonfinite, act, iters, final_norm);
}

// ---- general observation matrix (eq. error_forcing with a dense P_alpha; Alg. GTF-DEER) ----------
// The forcing is formed by k_obs_forced (z~_s = P_s z + alpha_s B^+ x_s, P_1 in the warm-up) into a
// forced-input array that the stored-Jacobian kernels read in place of their own diagonal forcing;
// the vanilla PLRNN runs through them as the shallow form with W2 = I, h2 = 0 (u = z~ exactly, so
// its ReLU decisions are those of z~).  J~_s = diag(A) P_s + W1 diag(m) (W2 P_s) is formed per step
// range (P_1 for s <= T_w, P_alpha after), then the dense scan solves the update; the warm-up is
// part of the one Newton iteration.
struct ObsWs {
    double *Bp64, *B64, *P164, *bgrad, *aug;
    float *Bp32, *Pa32, *P132, *Ca, *C1, *Id, *Va, *V1;
    float *Zt, *z0e;
    ShWs sh;
};

static ObsWs carve_obs(void *ws, const deer_model *m, const deer_forcing *f, int B, int T, int op, size_t *bytes) {
    const int M = m->M, N = f->n_forced, L = m->kind == DEER_SHPLRNN ? m->L : M;
    ObsWs w{};
    Carver c(ws);
    w.Bp64 = c.take<double>((size_t)M * N);
    w.B64 = c.take<double>((size_t)N * M);
    w.P164 = c.take<double>((size_t)M * M);
    w.aug = c.take<double>((size_t)64 * 128);
    w.Bp32 = c.take<float>((size_t)M * N);
    w.Pa32 = c.take<float>((size_t)M * M);
    w.P132 = c.take<float>((size_t)M * M);
    w.Ca = c.take<float>((size_t)M * M);
    w.C1 = c.take<float>((size_t)M * M);
    w.Id = c.take<float>((size_t)M * M);
    w.Va = c.take<float>((size_t)L * M);
    w.V1 = c.take<float>((size_t)L * M);
    w.Zt = c.take<float>((size_t)B * T * M);
    w.z0e = c.take<float>((size_t)B * M);
    if (op == DEER_OP_ADJOINT) w.bgrad = c.take<double>(obs_bgrad_ws_doubles(M, N));
    if (op == DEER_OP_JACOBIAN) {
        w.sh.masks = c.take<uint32_t>((size_t)B * T * ((L + 31) / 32));
        *bytes = c.off;
        return w;
    }
    size_t shb = 0;
    w.sh = carve_sh(ws ? (char *)ws + c.off : nullptr, B, T, M, L, op, true, true, &shb);
    *bytes = c.off + shb;
    return w;
}

static int obs_prepare(const deer_model *m, const deer_forcing *f, const ObsWs &w, hipStream_t st) {
    const bool sh = m->kind == DEER_SHPLRNN;
    ObsSetup s{f->obs, f->n_forced, m->M, sh ? m->L : m->M, f->alpha, m->A, sh ? m->W2 : nullptr,
               w.Bp64, w.B64, w.P164, w.Bp32, w.Pa32, w.P132, w.Ca, w.C1, w.Id, w.Va, w.V1, w.aug};
    return launch_obs_setup(s, st);
}

// J~ of every step into J: P_1 for the warm-up steps s = 0..T_w (step 0's Jacobian only multiplies
// Delta_0 = 0), P_alpha after; plain J_F (P = I) when unforced is set
static int obs_jacform(const deer_model *m, const deer_forcing *f, const ObsWs &w, int B, int T, const float *x,
                       const float *z0e, const uint32_t *masks, float *J, const int *active, const float *gamma,
                       bool unforced, hipStream_t st) {
    const bool sh = m->kind == DEER_SHPLRNN;
    const int L = sh ? m->L : m->M;
    ShArgs a{m->A, m->W, nullptr, m->h, sh ? m->h2 : nullptr, 0.f, 0, x, z0e, B, T, m->M, L};
    if (unforced) {
        a.W2 = sh ? m->W2 : w.Id;
        return launch_jacform_shplrnn(a, masks, J, active, gamma, st);
    }
    int rc;
    if (f->T_w > 0) {
        a.W2 = w.V1;
        a.Cd = w.C1;
        a.t_lo = 0;
        a.t_hi = f->T_w + 1;
        if ((rc = launch_jacform_shplrnn(a, masks, J, active, gamma, st))) return rc;
        if (f->T_w + 1 >= T) return DEER_OK;
        a.t_lo = f->T_w + 1;
        a.t_hi = T;
    }
    a.W2 = w.Va;
    a.Cd = w.Ca;
    return launch_jacform_shplrnn(a, masks, J, active, gamma, st);
}

static int solve_obs(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T,
                     const float *x, const float *z0, float *z, uint32_t *masks, int32_t *iters, float *final_norm,
                     void *ws, size_t ws_bytes, hipStream_t st) {
    int rc;
    const bool sh = m->kind == DEER_SHPLRNN;
    if (sh && (rc = check_shallow_limits(m))) return rc;
    const int M = m->M, N = f->n_forced, L = sh ? m->L : M;
    size_t need = 0;
    carve_obs(nullptr, m, f, B, T, DEER_OP_SOLVE, &need);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    ObsWs w = carve_obs(ws, m, f, B, T, DEER_OP_SOLVE, &need);
    if ((rc = obs_prepare(m, f, w, st))) return rc;
    if (o->init == DEER_INIT_TEACHER) {
        if ((rc = launch_obs_forced(1, nullptr, nullptr, nullptr, x, z0, w.Bp32, w.Pa32, w.P132, f->alpha, f->T_w, B, T,
                                    M, N, z, w.z0e, st)))
            return rc;
    } else if (o->init == DEER_INIT_ZERO) {
        if ((rc = launch_fill_f32(z, (size_t)B * T * M, 0.f, st))) return rc;
    }
    const float *z0e = z0 ? z0 : w.z0e;
    ShArgs ar{m->A, m->W, sh ? m->W2 : w.Id, m->h, sh ? m->h2 : nullptr, 0.f, 0, x, z0e, B, T, M, L};
    ar.zt = w.Zt;
    std::vector<int> act(B, 1), it(B, 0);
    std::vector<float> norm(B, NAN);
    bool nonfinite = false;
    const ShWs &s = w.sh;
    const DenseWs &d = s.d;
    auto update = [&](const int *dact, const float *gam, const int *zsel, float *zb, float *za, uint32_t *,
                      uint32_t) -> int {
        int r;
        if ((r = launch_obs_forced(0, zb, za, zsel, x, z0, w.Bp32, w.Pa32, w.P132, f->alpha, f->T_w, B, T, M, N, w.Zt,
                                   w.z0e, st)))
            return r;
        if ((r = launch_resjac_shplrnn(ar, zb, za, zsel, nullptr, s.r, s.masks, dact, st))) return r;
        if ((r = obs_jacform(m, f, w, B, T, x, z0e, s.masks, s.J, dact, gam, false, st))) return r;
        if ((r = launch_chunk_product_dense(false, B, T, M, s.J, s.r, -1.f, d.P, d.v, dact, d.C, d.ncs, st))) return r;
        if ((r = launch_carry(d.MP, false, d.P, d.v, d.carry, dact, nullptr, B, d.ncs, d.gws, st))) return r;
        return launch_fixup_dense(0, B, T, M, s.J, s.r, -1.f, d.carry, zb, za, zsel, s.ctl.chain_bits, dact, d.C,
                                  d.ncs, st);
    };
    if ((rc = newton_loop(o, B, (size_t)T * M, d.ncs, s.ctl, z, update, it, norm, nonfinite, act, st))) return rc;
    if (masks) {
        if ((rc = launch_obs_forced(0, z, nullptr, nullptr, x, z0, w.Bp32, w.Pa32, w.P132, f->alpha, f->T_w, B, T, M,
                                    N, w.Zt, w.z0e, st)))
            return rc;
        if ((rc = launch_resjac_shplrnn(ar, z, nullptr, nullptr, nullptr, nullptr, masks, nullptr, st))) return rc;
    }
    return finish_solve(o, B, it, norm, nonfinite, act, iters, final_norm);
}

static int jacobian_obs(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                        const float *z, float *F, float *r, float *J, uint32_t *masks, void *ws, size_t ws_bytes,
                        hipStream_t st) {
    int rc;
    const bool sh = m->kind == DEER_SHPLRNN;
    if (sh && (rc = check_shallow_limits(m))) return rc;
    const int M = m->M, N = f->n_forced, L = sh ? m->L : M;
    size_t need = 0;
    carve_obs(nullptr, m, f, B, T, DEER_OP_JACOBIAN, &need);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    ObsWs w = carve_obs(ws, m, f, B, T, DEER_OP_JACOBIAN, &need);
    if ((rc = obs_prepare(m, f, w, st))) return rc;
    if ((rc = launch_obs_forced(0, z, nullptr, nullptr, x, z0, w.Bp32, w.Pa32, w.P132, f->alpha, f->T_w, B, T, M, N,
                                w.Zt, w.z0e, st)))
        return rc;
    const float *z0e = z0 ? z0 : w.z0e;
    ShArgs ar{m->A, m->W, sh ? m->W2 : w.Id, m->h, sh ? m->h2 : nullptr, 0.f, 0, x, z0e, B, T, M, L};
    ar.zt = w.Zt;
    uint32_t *mk = masks ? masks : w.sh.masks;
    if ((rc = launch_resjac_shplrnn(ar, z, nullptr, nullptr, F, r, mk, nullptr, st))) return rc;
    if (J) return obs_jacform(m, f, w, B, T, x, z0e, mk, J, nullptr, nullptr, false, st);
    return DEER_OK;
}

static int adjoint_obs(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                       const float *z, const float *g, float *lam, const deer_grads *grads, void *ws, size_t ws_bytes,
                       hipStream_t st) {
    int rc;
    const bool sh = m->kind == DEER_SHPLRNN;
    if (sh && (rc = check_shallow_limits(m))) return rc;
    const int M = m->M, N = f->n_forced, L = sh ? m->L : M;
    size_t need = 0;
    carve_obs(nullptr, m, f, B, T, DEER_OP_ADJOINT, &need);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    ObsWs w = carve_obs(ws, m, f, B, T, DEER_OP_ADJOINT, &need);
    const ShWs &s = w.sh;
    const DenseWs &d = s.d;
    if ((rc = obs_prepare(m, f, w, st))) return rc;
    if ((rc = launch_obs_forced(0, z, nullptr, nullptr, x, z0, w.Bp32, w.Pa32, w.P132, f->alpha, f->T_w, B, T, M, N,
                                w.Zt, w.z0e, st)))
        return rc;
    const float *z0e = z0 ? z0 : w.z0e;
    ShArgs ar{m->A, m->W, sh ? m->W2 : w.Id, m->h, sh ? m->h2 : nullptr, 0.f, 0, x, z0e, B, T, M, L};
    ar.zt = w.Zt;
    if ((rc = launch_resjac_shplrnn(ar, z, nullptr, nullptr, nullptr, nullptr, s.masks, nullptr, st))) return rc;
    if ((rc = obs_jacform(m, f, w, B, T, x, z0e, s.masks, s.J, nullptr, nullptr, false, st))) return rc;
    const double mse_scale = 2.0 / ((double)B * N * (T - f->T_w));
    const float *gg = g;
    if (!gg) {
        if ((rc = launch_obs_seed(z, x, f->obs, (float)mse_scale, f->T_w, B, T, M, N, s.g, st))) return rc;
        gg = s.g;
    }
    float *lo = lam ? lam : s.lam;
    if ((rc = launch_chunk_product_dense(true, B, T, M, s.J, gg, 1.f, d.P, d.v, nullptr, d.C, d.ncs, st))) return rc;
    if ((rc = launch_carry(d.MP, true, d.P, d.v, d.carry, nullptr, nullptr, B, d.ncs, d.gws, st))) return rc;
    if ((rc = launch_fixup_dense(2, B, T, M, s.J, gg, 1.f, d.carry, nullptr, lo, nullptr, nullptr, nullptr, d.C, d.ncs,
                                 st)))
        return rc;
    if (!grads) return DEER_OK;
    if (grads->A || grads->W || grads->W2 || grads->h || grads->h2) {
        // the vanilla PLRNN as the shallow form: dW1 is dW, dh1 is dh, W2 = I and h2 are not parameters
        deer_grads gv{grads->A, grads->W, sh ? grads->W2 : nullptr, grads->h, sh ? grads->h2 : nullptr, nullptr};
        if ((rc = launch_grads_shplrnn(ar, z, lo, s.masks, s.part, &gv, st))) return rc;
    }
    if (grads->obs) {
        // mu_s = J_F(z~_s)^T lam_s needs the unforced Jacobians: formed into J (J~ is no longer used)
        if ((rc = obs_jacform(m, f, w, B, T, x, z0e, s.masks, s.J, nullptr, nullptr, true, st))) return rc;
        if ((rc = launch_obs_bgrad(s.J, lo, z, x, f->obs, w.Bp64, w.B64, w.P164, z0 != nullptr, f->alpha, f->T_w,
                                   g == nullptr, mse_scale, B, T, M, N, w.bgrad, grads->obs, st)))
            return rc;
    }
    return DEER_OK;
}

static int solve_quasi(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T,
                       const float *x, const float *z0, float *z, uint32_t *masks, int32_t *iters, float *final_norm,
                       void *ws, size_t ws_bytes, hipStream_t st) {
    size_t need = 0;
    const int L = quasi_L(m);
    carve_quasi(nullptr, B, T, m->M, L, DEER_OP_SOLVE, &need);
    int rc = check_ws(ws, ws_bytes, need);
    if (rc) return rc;
    QuasiWs w = carve_quasi(ws, B, T, m->M, L, DEER_OP_SOLVE, &need);
    PlrnnArgs a{m->A, m->W, m->h, f->alpha, f->n_forced, x, z0, B, T, m->M};
    ShArgs sa{m->A, m->W, m->W2, m->h, m->h2, f->alpha, f->n_forced, x, z0, B, T, m->M, m->L};
    a.tw = sa.tw = f->T_w;
    if ((rc = init_guess(o, B, T, m->M, f->n_forced, x, z, st))) return rc;
    std::vector<int> act(B, 1), it(B, 0);
    std::vector<float> norm(B, NAN);
    bool nonfinite = false;
    // vanilla PLRNN, adaptive loop: one kernel per pass (the fix-up of the previous update and
    // the chunk aggregates of the next, with the pass-end control)
    NewtonCtl ctl = w.ctl;
    const bool qf = L == 0 && o->fixed_iters <= 0 && (size_t)(T + 1) * m->M * 4 < ((size_t)1 << 31) &&
                    quasi_fusion_allowed();   // a sequence's rows addressed with 32-bit offsets
    if (qf) {
        ctl.fused = true;
        ctl.nd.pv = ctl.pv;
        ctl.lead = 1;
        uint32_t *mark_unused = nullptr;
        if ((rc = host_block(B, ctl.nd, &mark_unused))) return rc;
    }
    const FusedCtl fc{ctl.nd, ctl.seq, o->tol, o->step_bound == 0.f ? kDefaultStepBound : o->step_bound, kDamp};
    auto update = [&](const int *dact, const float *gam, const int *zsel, float *zb, float *za, uint32_t *mark,
                      uint32_t pass_no) -> int {
        if (qf) {   // aggregates alternate between the two sets
            const bool odd = pass_no & 1u;
            return launch_qdeer_pass(a, zb, za, odd ? w.P2 : w.P, odd ? w.v2 : w.v, odd ? w.gm2 : w.gm,
                                     odd ? w.P : w.P2, odd ? w.v : w.v2, odd ? w.gm : w.gm2, w.C, w.ncs, fc, mark,
                                     pass_no, st);
        }
        if (L == 0)
            return launch_qdeer_update(a, zb, za, zsel, dact, gam, w.rhs, w.coef, w.P, w.v, w.carry,
                                       w.ctl.chain_bits, w.C, w.ncs, st);
        // shallow: residual and hidden-unit masks, then the diagonal coefficients from the masks
        int r;
        if ((r = launch_resjac_shplrnn(sa, zb, za, zsel, nullptr, w.rhs, w.masks, dact, st))) return r;
        if ((r = launch_qdeer_shdiag(sa, w.masks, dact, gam, w.coef, st))) return r;
        return launch_qdeer_scan_fwd(B, T, m->M, x, f->n_forced, zb, za, zsel, dact, w.rhs, w.coef, w.P, w.v, w.carry,
                                     w.ctl.chain_bits, w.C, w.ncs, st);
    };
    if ((rc = newton_loop(o, B, (size_t)T * m->M, w.ncs, ctl, z, update, it, norm, nonfinite, act, st))) return rc;
    if (masks) {
        rc = L == 0 ? launch_resjac_plrnn(a, z, nullptr, nullptr, nullptr, masks, nullptr, st)
                    : launch_resjac_shplrnn(sa, z, nullptr, nullptr, nullptr, nullptr, masks, nullptr, st);
        if (rc) return rc;
    }
    return finish_solve(o, B, it, norm, nonfinite, act, iters, final_norm);
}

static size_t param_floats(const deer_model *m) {
    return m->kind == DEER_PLRNN ? (size_t)m->M * (m->M + 2) : (size_t)m->M * (2 * m->L + 2) + m->L;
}

static deer_grads grads_at(const deer_model *m, float *base) {
    deer_grads g{};
    const size_t M = m->M, L = m->L;
    g.A = base;
    if (m->kind == DEER_PLRNN) {
        g.W = base + M;
        g.h = base + M + M * M;
    } else {
        g.W = base + M;
        g.W2 = base + M + M * L;
        g.h = base + M + 2 * M * L;
        g.h2 = base + 2 * M + 2 * M * L;
    }
    return g;
}


}  // namespace deer

using namespace deer;

extern "C" {

const char *deer_status_string(int s) {
    switch (s) {
        case DEER_OK: return "ok";
        case DEER_ERR_INVALID_ARG: return "invalid argument";
        case DEER_ERR_NOT_CONVERGED: return "Newton iteration did not converge within max_iter";
        case DEER_ERR_NONFINITE: return "non-finite value in a Newton update";
        case DEER_ERR_HIP: return "HIP runtime error";
        case DEER_ERR_WORKSPACE: return "workspace too small or misaligned";
        default: return "unknown status";
    }
}

const char *deer_last_error(void) { return g_err; }

int deer_host_reserve(int max_batch) {
    set_error("");
    if (max_batch <= 0) { set_error("max_batch must be positive"); return DEER_ERR_INVALID_ARG; }
    return host_reserve(max_batch);
}

int deer_host_release(void) {
    set_error("");
    if (t_host.base) {
        hipError_t e = hipHostFree(t_host.base);
        t_host.base = nullptr;
        t_host.cap = 0;
        if (e != hipSuccess) return hip_fail(e, "hipHostFree");
    }
    return DEER_OK;
}

int deer_timing_enable(int on) {
    TimingState &s = tstate();
    std::lock_guard<std::mutex> g(s.mu);
    for (auto &kv : s.recs)
        for (auto &pr : kv.second) {
            s.pool.push_back(pr.first);
            s.pool.push_back(pr.second);
        }
    s.recs.clear();
    s.order.clear();
    s.on = on != 0;
    return DEER_OK;
}

int deer_timing_report(int idx, char *name, int name_cap, double *ms_total, long *launches) {
    TimingState &s = tstate();
    std::lock_guard<std::mutex> g(s.mu);
    const int n = (int)s.order.size();
    if (idx < 0 || idx >= n) return n;
    const std::string &k = s.order[idx];
    double tot = 0.0;
    for (auto &pr : s.recs[k]) {
        if (hipEventSynchronize(pr.second) != hipSuccess) return -DEER_ERR_HIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess) return -DEER_ERR_HIP;
        tot += ms;
    }
    if (name && name_cap > 0) {
        strncpy(name, k.c_str(), (size_t)name_cap - 1);
        name[name_cap - 1] = 0;
    }
    if (ms_total) *ms_total = tot;
    if (launches) *launches = (long)s.recs[k].size();
    return n;
}

size_t deer_workspace_bytes(const deer_model *m, int B, int T, int op) {
    deer_forcing f{0.f, 0};
    if (check_common(m, &f, B, T) != DEER_OK) return 0;
    if (op != DEER_OP_SOLVE && op != DEER_OP_ADJOINT) return 0;
    if (m->kind == DEER_DIAG_SSM) return diag_bytes(B, T, m->M, m->L, op);
    if (m->kind == DEER_PLRNN) {
        size_t bytes = 0;
        carve_plrnn(nullptr, B, T, m->M, op, &bytes);
        return bytes;
    }
    if (m->kind == DEER_SHPLRNN) {
        size_t bytes = 0;
        carve_sh(nullptr, B, T, m->M, m->L, op, true, true, &bytes, !sh_fused(m->M, m->L));
        return bytes;
    }
    return 0;
}

size_t deer_scan_workspace_bytes(int layout, int reverse, int transpose, int B, int T, int M) {
    (void)reverse;
    (void)transpose;
    if (B <= 0 || T <= 0 || M <= 0) return 0;
    if (layout == DEER_SCAN_DIAG_C64) return diag_scan_ws_bytes(B, T, M);
    if (layout == DEER_SCAN_DENSE && M <= 128) {
        size_t bytes = 0;
        carve_dense(nullptr, B, T, M, &bytes);
        return bytes;
    }
    return 0;
}

int plrnn_jacobian_ex(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                      const float *z, float *F, float *r, float *J, uint32_t *masks, void *ws, size_t ws_bytes,
                      void *stream) {
    set_error("");
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if (!f->obs) return plrnn_jacobian(m, f, B, T, x, z0, z, F, r, J, masks, stream);
    if (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN) {
        set_error("plrnn_jacobian_ex: PLRNN kinds only");
        return DEER_ERR_INVALID_ARG;
    }
    if (!x || !z) { set_error("x and z are required"); return DEER_ERR_INVALID_ARG; }
    return jacobian_obs(m, f, B, T, x, z0, z, F, r, J, masks, ws, ws_bytes, (hipStream_t)stream);
}

int plrnn_jacobian(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                   const float *z, float *F, float *r, float *J, uint32_t *masks, void *stream) {
    set_error("");
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if (f->T_w != 0) { set_error("plrnn_jacobian takes T_w = 0 (one forcing strength for every step)"); return DEER_ERR_INVALID_ARG; }
    if ((rc = no_obs(f, "plrnn_jacobian"))) return rc;
    if (!x || !z) { set_error("x and z are required"); return DEER_ERR_INVALID_ARG; }
    hipStream_t st = (hipStream_t)stream;
    if (m->kind == DEER_PLRNN) {
        PlrnnArgs a{m->A, m->W, m->h, f->alpha, f->n_forced, x, z0, B, T, m->M};
        return launch_resjac_plrnn(a, z, F, r, J, masks, nullptr, st);
    }
    if (m->kind == DEER_SHPLRNN) {
        if ((rc = check_shallow_limits(m))) return rc;
        ShArgs a{m->A, m->W, m->W2, m->h, m->h2, f->alpha, f->n_forced, x, z0, B, T, m->M, m->L};
        if ((rc = launch_resjac_shplrnn(a, z, nullptr, nullptr, F, r, masks, nullptr, st))) return rc;
        if (J) {
            if (!masks) { set_error("the shallow dense Jacobian output needs the masks output"); return DEER_ERR_INVALID_ARG; }
            if ((rc = launch_jacform_shplrnn(a, masks, J, nullptr, nullptr, st))) return rc;
        }
        return DEER_OK;
    }
    set_error("plrnn_jacobian: model kind %d not supported", m->kind);
    return DEER_ERR_INVALID_ARG;
}

int deer_solve(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T, const float *x,
               const float *z0, float *z, uint32_t *masks, int32_t *iters, float *final_norm, void *ws,
               size_t ws_bytes, void *stream) {
    set_error("");
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if (!o || !x || !z) { set_error("opts, x and z are required"); return DEER_ERR_INVALID_ARG; }
    if (o->init < 0 || o->init > 2) { set_error("unknown init %d", o->init); return DEER_ERR_INVALID_ARG; }
    if (!(o->tol >= 0.f) && o->fixed_iters <= 0) { set_error("tol must be >= 0"); return DEER_ERR_INVALID_ARG; }
    if (m->kind != DEER_DIAG_SSM && o->fixed_iters <= 0 && (rc = check_host_reserved(B))) return rc;
    hipStream_t st = (hipStream_t)stream;
    if (f->obs) return solve_obs(m, f, o, B, T, x, z0, z, masks, iters, final_norm, ws, ws_bytes, st);
    if (m->kind == DEER_PLRNN)
        return solve_plrnn(m, f, o, B, T, x, z0, z, masks, iters, final_norm, ws, ws_bytes, st);
    if (m->kind == DEER_SHPLRNN)
        return solve_shplrnn(m, f, o, B, T, x, z0, z, masks, iters, final_norm, ws, ws_bytes, st);
    if (m->kind == DEER_DIAG_SSM) {
        if ((rc = check_ws(ws, ws_bytes, diag_bytes(B, T, m->M, m->L, DEER_OP_SOLVE)))) return rc;
        rc = launch_diag_scan(false, B, T, m->M, m->A, nullptr, m->W, m->L, x, z, ws, st);
        if (rc) return rc;
        if (iters) for (int b = 0; b < B; ++b) iters[b] = 1;
        if (final_norm) for (int b = 0; b < B; ++b) final_norm[b] = 0.f;
        return DEER_OK;
    }
    set_error("deer_solve: model kind %d not supported yet", m->kind);
    return DEER_ERR_INVALID_ARG;
}

int deer_adjoint(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                 const float *z, const float *g, float *lam, const deer_grads *grads, void *ws, size_t ws_bytes,
                 void *stream) {
    return deer_adjoint_ex(m, f, B, T, x, z0, z, g, DEER_G_NATIVE, lam, grads, ws, ws_bytes, stream);
}

int deer_adjoint_ex(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                    const float *z, const float *g, int g_layout, float *lam, const deer_grads *grads, void *ws,
                    size_t ws_bytes, void *stream) {
    set_error("");
    if (g_layout != DEER_G_NATIVE && g_layout != DEER_G_REAL) {
        set_error("unknown cotangent layout %d", g_layout);
        return DEER_ERR_INVALID_ARG;
    }
    if (g_layout == DEER_G_REAL && m && m->kind != DEER_DIAG_SSM) {
        set_error("DEER_G_REAL applies to DEER_DIAG_SSM only");
        return DEER_ERR_INVALID_ARG;
    }
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if (!x || !z) { set_error("x and z are required"); return DEER_ERR_INVALID_ARG; }
    hipStream_t st = (hipStream_t)stream;
    if (f->obs) return adjoint_obs(m, f, B, T, x, z0, z, g, lam, grads, ws, ws_bytes, st);
    if (f->T_w > 0 && g_layout != DEER_G_NATIVE) {
        set_error("the latent warm-up takes the native cotangent layout");
        return DEER_ERR_INVALID_ARG;
    }
    if (m->kind == DEER_PLRNN) {
        size_t need = 0;
        carve_plrnn(nullptr, B, T, m->M, DEER_OP_ADJOINT, &need);
        if ((rc = check_ws(ws, ws_bytes, need))) return rc;
        PlrnnWs w = carve_plrnn(ws, B, T, m->M, DEER_OP_ADJOINT, &need);
        PlrnnArgs a{m->A, m->W, m->h, f->alpha, f->n_forced, x, z0, B, T, m->M};
        a.tw = f->T_w;   // > 0 only on the register-tiled path (M <= 16)
        // MSE seed over the states after the warm-up, z_{T_w+1}..z_T
        const float scale = f->n_forced > 0 ? (float)(2.0 / ((double)B * f->n_forced * (T - f->T_w))) : 0.f;
        if (a.tw == 0 && small_path_enabled() && adjoint_small_fits(m->M, T)) {   // one workgroup per sequence
            const bool gr = grads && (grads->A || grads->W || grads->h);
            if (B == 1)
                return launch_adjoint_small(a, g, scale, z, lam, nullptr, gr ? grads->A : nullptr,
                                            gr ? grads->W : nullptr, gr ? grads->h : nullptr, st);
            if ((rc = launch_adjoint_small(a, g, scale, z, lam, w.gpart, nullptr, nullptr, nullptr, st))) return rc;
            if (gr) return launch_reduce_gpart(w.gpart, B, 4, m->M, grads->A, grads->W, grads->h, w.gpart2, st);
            return DEER_OK;
        }
        if (w.MP == 16) {   // register-tiled path: masks from z inside the kernels, per-wave gradients
            if ((rc = launch_adjoint_plrnn16(a, g, scale, z, w.P, w.v, w.carry, lam, w.gpart, w.C, w.ncs, st)))
                return rc;
            if (grads && (grads->A || grads->W || grads->h)) {
                if ((rc = launch_reduce_gpart(w.gpart, (B * w.ncs + 3) / 4, 16, m->M, grads->A, grads->W, grads->h,
                                              w.gpart2, st)))
                    return rc;
            }
            return DEER_OK;
        }
        if ((rc = launch_resjac_plrnn(a, z, nullptr, nullptr, nullptr, w.masks, nullptr, st))) return rc;
        if ((rc = launch_chunk_product_plrnn(a, true, w.masks, g, z, scale, w.P, w.v, nullptr, w.C, w.ncs, st)))
            return rc;
        if ((rc = launch_carry(w.MP, true, w.P, w.v, w.carry, nullptr, nullptr, B, w.ncs, w.gws, st))) return rc;
        if ((rc = launch_fixup_rev_plrnn(a, w.masks, g, scale, z, w.carry, lam, w.gpart, w.C, w.ncs, st))) return rc;
        if (grads && (grads->A || grads->W || grads->h)) {
            if ((rc = launch_reduce_gpart(w.gpart, B * w.ncs, w.MP, m->M, grads->A, grads->W, grads->h, w.gpart2, st))) return rc;
        }
        return DEER_OK;
    }
    if (m->kind == DEER_SHPLRNN) {
        if ((rc = check_shallow_limits(m))) return rc;
        const bool fused = sh_fused(m->M, m->L);
        size_t need = 0;
        carve_sh(nullptr, B, T, m->M, m->L, DEER_OP_ADJOINT, true, true, &need, !fused);
        if ((rc = check_ws(ws, ws_bytes, need))) return rc;
        ShWs w = carve_sh(ws, B, T, m->M, m->L, DEER_OP_ADJOINT, true, true, &need, !fused);
        ShArgs a{m->A, m->W, m->W2, m->h, m->h2, f->alpha, f->n_forced, x, z0, B, T, m->M, m->L};
        a.tw = f->T_w;
        const DenseWs &d = w.d;
        const float *gg = g;
        if (!gg) {   // MSE over the states after the warm-up, z_{T_w+1}..z_T
            const float scale = f->n_forced > 0 ? (float)(2.0 / ((double)B * f->n_forced * (T - f->T_w))) : 0.f;
            if ((rc = launch_mse_seed(z, x, scale, B, T, m->M, f->n_forced, w.g, st, f->T_w))) return rc;
            gg = w.g;
        }
        float *lo = lam ? lam : w.lam;
        if ((rc = launch_resjac_shplrnn(a, z, nullptr, nullptr, nullptr, nullptr, w.masks, nullptr, st))) return rc;
        if (fused) {
            if ((rc = launch_chunk_product_shfused(true, a, w.masks, gg, 1.f, nullptr, d.P, d.v, nullptr, d.C, d.ncs,
                                                   st)))
                return rc;
            if ((rc = launch_carry(d.MP, true, d.P, d.v, d.carry, nullptr, nullptr, B, d.ncs, d.gws, st))) return rc;
            if ((rc = launch_fixup_shjvp(true, a, w.masks, gg, 1.f, nullptr, d.carry, nullptr, lo, nullptr, nullptr,
                                         nullptr, d.C, d.ncs, st)))
                return rc;
        } else {
            if ((rc = jacform_sh(a, w.masks, w.J, nullptr, nullptr, st))) return rc;
            if ((rc = launch_chunk_product_dense(true, B, T, m->M, w.J, gg, 1.f, d.P, d.v, nullptr, d.C, d.ncs, st)))
                return rc;
            if ((rc = launch_carry(d.MP, true, d.P, d.v, d.carry, nullptr, nullptr, B, d.ncs, d.gws, st))) return rc;
            if ((rc = launch_fixup_dense(2, B, T, m->M, w.J, gg, 1.f, d.carry, nullptr, lo, nullptr, nullptr, nullptr,
                                         d.C, d.ncs, st)))
                return rc;
        }
        if (grads && (grads->A || grads->W || grads->W2 || grads->h || grads->h2)) {
            if ((rc = launch_grads_shplrnn(a, z, lo, w.masks, w.part, grads, st))) return rc;
        }
        return DEER_OK;
    }
    if (m->kind == DEER_DIAG_SSM) {
        if (!g) { set_error("DIAG_SSM adjoint needs the cotangent g"); return DEER_ERR_INVALID_ARG; }
        if ((rc = check_ws(ws, ws_bytes, diag_bytes(B, T, m->M, m->L, DEER_OP_ADJOINT)))) return rc;
        float *dlam = grads ? grads->A : nullptr, *dBc = grads ? grads->W : nullptr;
        if (!lam && !dlam && !dBc) return DEER_OK;
        return launch_diag_adjoint(B, T, m->M, m->L, m->A, g, g_layout == DEER_G_REAL, z, x, lam, dlam, dBc, ws, st);
    }
    set_error("deer_adjoint: model kind %d not supported yet", m->kind);
    return DEER_ERR_INVALID_ARG;
}

int deer_solve_quasi(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, int B, int T,
                     const float *x, const float *z0, float *z, uint32_t *masks, int32_t *iters, float *final_norm,
                     void *ws, size_t ws_bytes, void *stream) {
    set_error("");
    int rc = check_quasi(m, f, B, T);
    if (rc) return rc;
    if (!o || !x || !z) { set_error("opts, x and z are required"); return DEER_ERR_INVALID_ARG; }
    if (o->init < 0 || o->init > 2) { set_error("unknown init %d", o->init); return DEER_ERR_INVALID_ARG; }
    if (!(o->tol >= 0.f) && o->fixed_iters <= 0) { set_error("tol must be >= 0"); return DEER_ERR_INVALID_ARG; }
    if (o->fixed_iters <= 0 && (rc = check_host_reserved(B))) return rc;
    return solve_quasi(m, f, o, B, T, x, z0, z, masks, iters, final_norm, ws, ws_bytes, (hipStream_t)stream);
}

int deer_adjoint_quasi(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0,
                       const float *z, const float *g, float *lam, const deer_grads *grads, void *ws, size_t ws_bytes,
                       void *stream) {
    set_error("");
    int rc = check_quasi(m, f, B, T);
    if (rc) return rc;
    if (!x || !z) { set_error("x and z are required"); return DEER_ERR_INVALID_ARG; }
    hipStream_t st = (hipStream_t)stream;
    size_t need = 0;
    const int L = quasi_L(m);
    carve_quasi(nullptr, B, T, m->M, L, DEER_OP_ADJOINT, &need);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    QuasiWs w = carve_quasi(ws, B, T, m->M, L, DEER_OP_ADJOINT, &need);
    PlrnnArgs a{m->A, m->W, m->h, f->alpha, f->n_forced, x, z0, B, T, m->M};
    a.tw = f->T_w;
    // MSE over the states after the latent warm-up, z_{T_w+1}..z_T
    const float scale = f->n_forced > 0 ? (float)(2.0 / ((double)B * f->n_forced * (T - f->T_w))) : 0.f;
    if (L > 0) {
        // shallow: masks and coefficients at z, the reverse scan writes lam, then the shallow
        // gradient kernel (dA, dW1, dW2, dh1, dh2) from it
        ShArgs sa{m->A, m->W, m->W2, m->h, m->h2, f->alpha, f->n_forced, x, z0, B, T, m->M, m->L};
        sa.tw = f->T_w;
        float *lo = lam ? lam : w.lam;
        if ((rc = launch_resjac_shplrnn(sa, z, nullptr, nullptr, nullptr, nullptr, w.masks, nullptr, st))) return rc;
        if ((rc = launch_qdeer_shdiag(sa, w.masks, nullptr, nullptr, w.coef, st))) return rc;
        if ((rc = launch_qdeer_scan_rev(a, g, scale, z, w.coef, w.P, w.v, w.carry, lo, nullptr, w.C, w.ncs, st)))
            return rc;
        if (grads && (grads->A || grads->W || grads->W2 || grads->h || grads->h2))
            return launch_grads_shplrnn(sa, z, lo, w.masks, w.part, grads, st);
        return DEER_OK;
    }
    if ((rc = launch_qdeer_adjoint(a, g, scale, z, w.coef, w.P, w.v, w.carry, lam, w.gpart, w.C, w.ncs, st))) return rc;
    if (grads && (grads->A || grads->W || grads->h))
        return launch_reduce_gpart(w.gpart, B * w.ncs, w.MP, m->M, grads->A, grads->W, grads->h, w.gpart2, st);
    return DEER_OK;
}

size_t deer_workspace_bytes_ex(const deer_model *m, const deer_forcing *f, int B, int T, int op, int quasi) {
    if (f && f->obs) {
        if (quasi || check_common(m, f, B, T) != DEER_OK) return 0;
        if (op != DEER_OP_SOLVE && op != DEER_OP_ADJOINT && op != DEER_OP_JACOBIAN) return 0;
        if (m->kind == DEER_SHPLRNN && check_shallow_limits(m) != DEER_OK) return 0;
        size_t bytes = 0;
        carve_obs(nullptr, m, f, B, T, op, &bytes);
        return bytes;
    }
    // a latent warm-up is part of the one Newton iteration: the workspace of the plain solve
    if (f && f->T_w > 0 && (quasi ? check_quasi(m, f, B, T) : check_common(m, f, B, T)) != DEER_OK) return 0;
    return quasi ? deer_quasi_workspace_bytes(m, B, T, op) : deer_workspace_bytes(m, B, T, op);
}

size_t deer_train_params(const deer_model *m) {
    if (!m || (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN)) return 0;
    return param_floats(m);
}

size_t deer_train_workspace_bytes(const deer_model *m, const deer_forcing *f, int B, int T, int quasi) {
    const size_t a = deer_workspace_bytes_ex(m, f, B, T, DEER_OP_SOLVE, quasi);
    const size_t b = deer_workspace_bytes_ex(m, f, B, T, DEER_OP_ADJOINT, quasi);
    if (!a || !b || (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN)) return 0;
    Carver c(nullptr);
    c.take<float>(param_floats(m));
    c.take<double>(train_partials() + 1);
    c.take<char>(a > b ? a : b);
    return c.off;
}

int deer_train_step(const deer_model *m, const deer_forcing *f, const deer_solve_opts *o, const deer_train_opts *tr,
                    int B, int T, const float *x, const float *z0, float *z, float *adam_m, float *adam_v,
                    const deer_grads *grads_out, float *loss, int32_t *iters, void *ws, size_t ws_bytes,
                    void *stream) {
    set_error("");
    int rc = check_common(m, f, B, T);
    if (rc) return rc;
    if (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN) { set_error("deer_train_step: PLRNN kinds only"); return DEER_ERR_INVALID_ARG; }
    if (!o || !tr || !x || !z || !adam_m || !adam_v) { set_error("opts, train, x, z and the Adam moments are required"); return DEER_ERR_INVALID_ARG; }
    if (o->fixed_iters > 0) { set_error("deer_train_step solves to a tolerance (fixed_iters = 0)"); return DEER_ERR_INVALID_ARG; }
    if ((rc = no_obs(f, "deer_train_step"))) return rc;
    if ((rc = check_host_reserved(B))) return rc;
    if (tr->step < 1 || !(tr->lr > 0.f) || !(tr->beta1 >= 0.f && tr->beta1 < 1.f) || !(tr->beta2 >= 0.f && tr->beta2 < 1.f)) {
        set_error("Adam needs step >= 1, lr > 0 and betas in [0, 1)");
        return DEER_ERR_INVALID_ARG;
    }
    if (tr->mar_lambda != 0.f && (tr->mar_units < 1 || tr->mar_units > m->M || (tr->mar_p != 1 && tr->mar_p != 2))) {
        set_error("MAR needs 1 <= mar_units <= M and mar_p in {1, 2}");
        return DEER_ERR_INVALID_ARG;
    }
    if (f->n_forced < 1) { set_error("the MSE needs at least one observed latent (n_forced >= 1)"); return DEER_ERR_INVALID_ARG; }
    const bool quasi = tr->quasi != 0;
    const size_t need = deer_train_workspace_bytes(m, f, B, T, tr->quasi);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    hipStream_t st = (hipStream_t)stream;
    Carver c(ws);
    float *g = c.take<float>(param_floats(m));
    double *part = c.take<double>(train_partials() + 1);
    const size_t a = deer_workspace_bytes_ex(m, f, B, T, DEER_OP_SOLVE, tr->quasi);
    const size_t b = deer_workspace_bytes_ex(m, f, B, T, DEER_OP_ADJOINT, tr->quasi);
    const size_t inner_bytes = a > b ? a : b;
    void *inner = c.take<char>(inner_bytes);
    // the solve, then the gradient of the MSE at its result (the adjoint's own MSE seed)
    rc = (quasi ? deer_solve_quasi : deer_solve)(m, f, o, B, T, x, z0, z, nullptr, iters, nullptr, inner, inner_bytes,
                                                 stream);
    if (rc) return rc;
    const deer_grads gbuf = grads_at(m, g);
    rc = (quasi ? deer_adjoint_quasi : deer_adjoint)(m, f, B, T, x, z0, z, nullptr, nullptr, &gbuf, inner,
                                                     inner_bytes, stream);
    if (rc) return rc;
    if (!m->h) {   // untrained (absent) biases: zero gradients so the layout stays uniform
        if ((rc = launch_fill_f32(gbuf.h, m->M, 0.f, st))) return rc;
    }
    if (m->kind == DEER_SHPLRNN && !m->h2) {
        if ((rc = launch_fill_f32(gbuf.h2, m->L, 0.f, st))) return rc;
    }
    const bool sh = m->kind == DEER_SHPLRNN;
    double *mar = part + train_partials();
    const bool with_mar = tr->mar_lambda != 0.f;
    if (with_mar && (rc = launch_mar(sh, m->A, m->W, sh ? m->W2 : nullptr, m->h, m->M, sh ? m->L : m->M,
                                     tr->mar_units, tr->mar_lambda, tr->mar_p, tr->mar_gamma_w, tr->mar_gamma_v, g,
                                     mar, st)))
        return rc;
    if (loss) {
        if ((rc = launch_mse_loss_partial(z, x, B, T, m->M, f->n_forced, f->T_w, part, st))) return rc;
        const double scale = 1.0 / ((double)B * f->n_forced * (T - f->T_w));
        if ((rc = launch_loss_final(part, scale, with_mar ? mar : nullptr, loss, st))) return rc;
    }
    if (grads_out) {
        const size_t M = m->M, L = m->L;
        const float *src[5] = {gbuf.A, gbuf.W, gbuf.W2, gbuf.h, gbuf.h2};
        float *dst[5] = {grads_out->A, grads_out->W, sh ? grads_out->W2 : nullptr, grads_out->h,
                         sh ? grads_out->h2 : nullptr};
        const size_t n[5] = {M, sh ? M * L : M * M, L * M, M, L};
        for (int k = 0; k < 5; ++k)
            if (dst[k]) DEER_HIP(hipMemcpyAsync(dst[k], src[k], n[k] * sizeof(float), hipMemcpyDeviceToDevice, st));
    }
    // Adam on the parameters in place
    const long M = m->M, L = m->L;
    float *params[5] = {const_cast<float *>(m->A), const_cast<float *>(m->W), sh ? const_cast<float *>(m->W2) : nullptr,
                        const_cast<float *>(m->h), sh ? const_cast<float *>(m->h2) : nullptr};
    const long sizes[5] = {M, sh ? M * L : M * M, sh ? L * M : 0, M, sh ? L : 0};
    return launch_adam(params, sizes, g, adam_m, adam_v, tr->lr, tr->beta1, tr->beta2, tr->eps, tr->step, st);
}

size_t deer_quasi_workspace_bytes(const deer_model *m, int B, int T, int op) {
    deer_forcing f{0.f, 0};
    if (check_quasi(m, &f, B, T) != DEER_OK) return 0;
    if (op != DEER_OP_SOLVE && op != DEER_OP_ADJOINT) return 0;
    size_t bytes = 0;
    carve_quasi(nullptr, B, T, m->M, quasi_L(m), op, &bytes);
    return bytes;
}

static int check_readout(const deer_readout *r, int B, int T, int M) {
    if (!r || !r->Wa || !r->Wb) { set_error("read-out needs Wa and Wb"); return DEER_ERR_INVALID_ARG; }
    if (B <= 0 || T <= 0) { set_error("B and T must be positive"); return DEER_ERR_INVALID_ARG; }
    if (M <= 0 || M > 64) { set_error("read-out supports 1 <= M <= 64 (M=%d)", M); return DEER_ERR_INVALID_ARG; }
    if (r->H <= 0 || r->H > 128) { set_error("read-out supports 1 <= H <= 128 (H=%d)", r->H); return DEER_ERR_INVALID_ARG; }
    if (r->n_out <= 0 || r->n_out > 4) { set_error("read-out supports 1 <= n_out <= 4"); return DEER_ERR_INVALID_ARG; }
    if ((long)B * (long)T > (1L << 31)) { set_error("B*T too large"); return DEER_ERR_INVALID_ARG; }
    return DEER_OK;
}

// ---- sequential baseline -------------------------------------------------------------------
static int check_sequential(const deer_model *m, const deer_forcing *f, int B, int T, SeqArgs *a) {
    if (!m || !f) { set_error("model/forcing pointer is NULL"); return DEER_ERR_INVALID_ARG; }
    if (no_obs(f, "deer_sequential")) return DEER_ERR_INVALID_ARG;
    if (m->kind != DEER_PLRNN && m->kind != DEER_SHPLRNN) {
        set_error("the sequential baseline covers the PLRNN kinds");
        return DEER_ERR_INVALID_ARG;
    }
    if (B <= 0 || T <= 0) { set_error("B and T must be positive (B=%d, T=%d)", B, T); return DEER_ERR_INVALID_ARG; }
    if (!(f->alpha >= 0.0f && f->alpha <= 1.0f)) { set_error("alpha must lie in [0, 1]"); return DEER_ERR_INVALID_ARG; }
    if (m->M <= 0 || f->n_forced < 0 || f->n_forced > m->M) {
        set_error("need M >= 1 and 0 <= n_forced <= M");
        return DEER_ERR_INVALID_ARG;
    }
    if (!m->A || !m->W || (m->kind == DEER_SHPLRNN && (!m->W2 || m->L <= 0))) {
        set_error("model parameters A, W (and W2, L for the shallow kind) are required");
        return DEER_ERR_INVALID_ARG;
    }
    const bool sh = m->kind == DEER_SHPLRNN;
    const int L = sh ? m->L : m->M;
    if (seq_check(m->M, L, sh)) {
        set_error("the sequential baseline supports M, L <= 256 and M L <= 8192 (M=%d, L=%d)", m->M, L);
        return DEER_ERR_INVALID_ARG;
    }
    if ((long)B * (long)T * (m->M > L ? m->M : L) >= (1L << 31)) { set_error("B*T too large"); return DEER_ERR_INVALID_ARG; }
    *a = SeqArgs{m->A, m->W, sh ? m->W2 : nullptr, m->h, sh ? m->h2 : nullptr, f->alpha, f->n_forced, nullptr,
                 nullptr, B, T, m->M, L, sh};
    return DEER_OK;
}

static void carve_seq(void *ws, const SeqArgs &a, float **act, float **part, size_t *bytes) {
    Carver c(ws);
    *act = a.sh ? c.take<float>((size_t)a.B * a.T * a.L) : nullptr;
    *part = c.take<float>((size_t)a.B * seq_part_floats(a.M, a.L, a.sh));
    *bytes = c.off;
}

size_t deer_readout_workspace_bytes(const deer_readout *r, int B, int T, int M) {
    if (check_readout(r, B, T, M) != DEER_OK) return 0;
    return readout_ws_bytes(B, T);
}

int deer_readout_loss(const deer_readout *r, int B, int T, int M, const float *h, const float *x, float *g,
                      float *loss, uint32_t *masks, const deer_readout_grads *grads, void *ws, size_t ws_bytes,
                      void *stream) {
    set_error("");
    int rc = check_readout(r, B, T, M);
    if (rc) return rc;
    if (!h || !x || !g) { set_error("h, x and g are required"); return DEER_ERR_INVALID_ARG; }
    if ((rc = check_ws(ws, ws_bytes, readout_ws_bytes(B, T)))) return rc;
    RoArgs ra{r->Wa, r->ca, r->Wb, r->cb, M, r->H, r->n_out};
    RoGrads gr{grads ? grads->Wa : nullptr, grads ? grads->ca : nullptr, grads ? grads->Wb : nullptr,
               grads ? grads->cb : nullptr};
    return launch_readout(ra, B, T, h, x, g, masks, loss, gr, ws, (hipStream_t)stream);
}

int deer_scan(int layout, int reverse, int transpose, int B, int T, int M, const float *J, const float *b, float *y,
              void *ws, size_t ws_bytes, void *stream) {
    set_error("");
    if (B <= 0 || T <= 0 || M <= 0) { set_error("B, T, M must be positive"); return DEER_ERR_INVALID_ARG; }
    if (!J || !b || !y) { set_error("J, b and y are required"); return DEER_ERR_INVALID_ARG; }
    if (b == y) { set_error("y may not alias b"); return DEER_ERR_INVALID_ARG; }
    hipStream_t st = (hipStream_t)stream;
    const bool rev = reverse != 0, tr = transpose != 0;
    if (layout == DEER_SCAN_DIAG_C64) {
        int rc = check_ws(ws, ws_bytes, diag_scan_ws_bytes(B, T, M));
        if (rc) return rc;
        // the transpose of multiplication by lambda (C read as R^2) is multiplication by conj(lambda)
        return launch_diag_scan(rev, B, T, M, J, b, nullptr, 0, nullptr, y, ws, st, tr ? 1 : 0);
    }
    if (layout == DEER_SCAN_DENSE) {
        if (M > 128) { set_error("dense scans support M <= 128"); return DEER_ERR_INVALID_ARG; }
        size_t need = 0;
        carve_dense(nullptr, B, T, M, &need);
        int rc = check_ws(ws, ws_bytes, need);
        if (rc) return rc;
        DenseWs w = carve_dense(ws, B, T, M, &need);
        // the kernels' default orientation is J_t forward and J_{t+1}^T in reverse
        const bool flip = tr != rev;
        if ((rc = launch_chunk_product_dense(rev, B, T, M, J, b, 1.f, w.P, w.v, nullptr, w.C, w.ncs, st, flip)))
            return rc;
        if ((rc = launch_carry(w.MP, rev, w.P, w.v, w.carry, nullptr, nullptr, B, w.ncs, w.gws, st))) return rc;
        return launch_fixup_dense(rev ? 2 : 1, B, T, M, J, b, 1.f, w.carry, nullptr, y, nullptr, nullptr, nullptr, w.C,
                                  w.ncs, st, flip);
    }
    set_error("deer_scan: unknown layout %d", layout);
    return DEER_ERR_INVALID_ARG;
}

size_t deer_sequential_workspace_bytes(const deer_model *m, int B, int T) {
    deer_forcing f{0.f, 0};
    SeqArgs a{};
    if (check_sequential(m, &f, B, T, &a)) return 0;
    float *act = nullptr, *part = nullptr;
    size_t need = 0;
    carve_seq(nullptr, a, &act, &part, &need);
    return need;
}

int deer_sequential(const deer_model *m, const deer_forcing *f, int B, int T, const float *x, const float *z0, float *z,
                    const float *g, float *lam, const deer_grads *grads, void *ws, size_t ws_bytes, void *stream) {
    set_error("");
    if (f && f->T_w != 0) { set_error("the sequential baseline runs without warm-up (T_w = 0)"); return DEER_ERR_INVALID_ARG; }
    SeqArgs a{};
    int rc = check_sequential(m, f, B, T, &a);
    if (rc) return rc;
    if (!x || !z) { set_error("x and z are required"); return DEER_ERR_INVALID_ARG; }
    a.x = x;
    a.z0 = z0;
    float *act = nullptr, *part = nullptr;
    size_t need = 0;
    carve_seq(nullptr, a, &act, &part, &need);
    if ((rc = check_ws(ws, ws_bytes, need))) return rc;
    carve_seq(ws, a, &act, &part, &need);
    hipStream_t st = (hipStream_t)stream;
    const bool back = lam || (grads && (grads->A || grads->W || grads->W2 || grads->h || grads->h2));
    if ((rc = launch_seq_forward(a, z, back ? act : nullptr, st))) return rc;
    if (!back) return DEER_OK;
    const float scale = f->n_forced > 0 ? (float)(2.0 / ((double)B * f->n_forced * T)) : 0.f;
    return launch_seq_backward(a, z, act, g, scale, lam, part, grads, st);
}

}  // extern "C"
