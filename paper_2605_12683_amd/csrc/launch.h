// Internal launcher interface between the C-ABI layer and the kernel translation units.
#pragma once
#include "common.h"

namespace deer {

struct FusedCtl;   // pass-end control fused into a pass kernel (defined below)

struct PlrnnArgs {
    const float *A, *W, *h;
    float alpha;
    int N;
    const float *x, *z0;
    int B, T, M;
    // latent warm-up inside the Newton iteration (M <= 16 kernels and the mask pass): the forced
    // inputs of steps 1..tw take alpha = 1 and their Jacobians P_1; 0 = none
    int tw = 0;
};

struct ShArgs {
    const float *A, *W1, *W2, *h1, *h2;
    float alpha;
    int N;
    const float *x, *z0;
    int B, T, M, L;
    // general observation matrix (the forcing is formed outside these kernels; alpha = N = 0):
    //   zt     [B,T,M]: zt[b, s] is the forced input z~_s of step s + 1 for s >= 1 (row 0 unused;
    //          z~_0 = z0), read instead of forming it from z and x (residual, gradients)
    //   Cd     [M,M]: dense term of the forced Jacobian, J~ = Cd + W1 diag(m) W2, replacing the
    //          diagonal diag(A) P (Jacobian formation; W2 is then W2 P)
    //   t_lo, t_hi: the Jacobian formation covers steps t_lo <= s < t_hi only (t_hi = 0: all)
    const float *zt = nullptr;
    const float *Cd = nullptr;
    int t_lo = 0, t_hi = 0;
    // latent warm-up inside the Newton iteration (identity read-out): the forced inputs of steps
    // 1..tw take alpha = 1 and the Jacobians of those steps P_1; 0 = none.  The stored-Jacobian
    // formation takes the warm-up as a separate step range with alpha = 1 instead.
    int tw = 0;
};

int padded_dim(int M);

// vanilla PLRNN
int launch_resjac_plrnn(const PlrnnArgs &a, const float *z, float *F, float *r, float *J, uint32_t *masks,
                        const int *active, hipStream_t st);
int launch_chunk_product_plrnn(const PlrnnArgs &a, bool rev, const uint32_t *masks, const float *rhs, const float *z,
                               float seed_scale, float *P, float *v, const int *active, int C, int ncs,
                               hipStream_t st);
// M <= 16 only: block 0 of the pass writes pass_no to the host-visible word *mark as it
// starts (every kernel queued before it has completed); mark may be null
int launch_newton_product_plrnn(const PlrnnArgs &a, const float *z, const float *zalt, const int *zsel, float *r,
                                uint32_t *masks, float *P, float *v, const int *active, const float *gamma, int C,
                                int ncs, int wmaps, float *gmap, uint32_t *mark, uint32_t pass_no, hipStream_t st);
// M <= 16 with wave maps (P, v from launch_newton_product_plrnn with wmaps): carries of the
// wave maps, written to the carry slot of each wave's first chunk
int launch_carry_walk16(bool rev, const float *P, const float *v, float *carry, const int *active, int B, int ncs,
                        hipStream_t st);
// M <= 16 adjoint: reverse chunk products (masks formed from z), carries, reverse fix-up with
// the gradient partials of each wave of four chains (gpart[(B ncs + 3) / 4][16][18])
int launch_adjoint_plrnn16(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *P, float *v,
                           float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st);
int launch_carry(int MP, bool rev, const float *P, const float *v, float *carry_in, const int *active,
                 uint32_t *norm_bits, int B, int ncs, float *gws, hipStream_t st);
size_t carry_ws_floats(int MP, int B, int ncs);
int launch_fixup_fwd_plrnn(const PlrnnArgs &a, const uint32_t *masks, const float *r, const float *carry_in,
                           float *z, float *zalt, const int *zsel, uint32_t *chain_bits, const int *active,
                           const float *gamma, int C, int ncs, const float *Pm, const float *vm,
                           const float *gmap, const FusedCtl *fc, hipStream_t st);
// device-side Newton control (one entry per sequence)
struct NewtonDev {
    int *act;       // active flag (read by every kernel of a pass)
    float *gamma;   // damping of the linearisation
    int *sel;       // which iterate buffer holds the current iterate
    float *om;      // 1 - gamma
    int *it;        // accepted updates
    float *norm;    // max |Delta| of the last accepted (or final) update
    int *status;    // 0 running, 1 converged, 2 non-finite
    // pinned host block (all four may be null): when a sequence stops, its update count,
    // last max |Delta| and status are written to hit, hnorm, hstat, and then (with release
    // order at system scope) its entry of hact, set to 1 by the host, is cleared
    int *hact;
    int *hit;
    float *hnorm;
    int *hstat;
    // fused passes only (else null): number of the pass whose kernel may use the chunk
    // aggregates stored for the sequence's current iterate (see launch_newton_pass16)
    uint32_t *pv;
};
struct NewtonDamp {
    float first, grow, shrink, floor;
};
int launch_seq_ctl(const uint32_t *chain_bits, const NewtonDev &nd, int B, int ncs, float tol, float bound,
                   const NewtonDamp &dp, hipStream_t st);
// The pass-end control of k_seq_ctl taken by the fix-up itself: per sequence a 96-word block of
// seq (arrival count, max |Delta| bits, max |z| bits, one 128-byte line each) is updated with device-scope atomics and the
// last chain of the sequence to arrive takes the decision.  seq == nullptr: not fused.
struct FusedCtl {
    NewtonDev nd;
    uint32_t *seq;
    float tol, bound;
    NewtonDamp dp;
};
constexpr int kSeqWords = 96;
// One kernel per Newton pass (M <= 16, adaptive loop, every sequence a whole number of blocks of
// 32 chunks of C steps, C a multiple of 16): the fix-up of the previous pass from the aggregates
// in (Pin, vin, gin), where fc.nd.pv says they belong to the current iterate, then the forward
// pass of the next update on the new iterate, its aggregates written to (Pout, vout, gout).
// Block 0 writes pass_no to *mark as it starts.
int launch_newton_pass16(const PlrnnArgs &a, float *z, float *zalt, const float *Pin, const float *vin,
                         const float *gin, float *Pout, float *vout, float *gout, int C, int ncs, const FusedCtl &fc,
                         uint32_t *mark, uint32_t pass_no, hipStream_t st);
int launch_ctl_init(const NewtonDev &nd, uint32_t *seq, int B, hipStream_t st);
int launch_seq_max(const uint32_t *chain_bits, const int *active, uint32_t *norm_bits, int B, int ncs,
                   hipStream_t st);
int launch_fixup_rev_plrnn(const PlrnnArgs &a, const uint32_t *masks, const float *g, float seed_scale, const float *z,
                           const float *carry_in, float *lam, float *gpart, int C, int ncs, hipStream_t st);
int launch_reduce_gpart(const float *gpart, int nchains, int MP, int M, float *dA, float *dW, float *dh,
                        double *part2, hipStream_t st);
size_t reduce_gpart_ws_bytes(int MP);

// small vanilla PLRNNs (M <= 4, T <= 4096) with a fixed number of plain Newton updates: the
// whole solve in one launch (one workgroup per sequence, update in place); norm_bits[b] gets
// max |Delta| of the last update
bool newton_small_fits(int M, int T, int fixed_iters);
int launch_newton_small(const PlrnnArgs &a, float *z, int iters, uint32_t *norm_bits, hipStream_t st);
// adjoint and gradient partials of M <= 4, T <= 4096 in one launch per batch: gpart[b][4][6]
// (MP = 4 for launch_reduce_gpart); with gpart null the gradients of the single sequence go to
// dA / dW / dh directly (B = 1)
bool adjoint_small_fits(int M, int T);
int launch_adjoint_small(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *lam,
                         float *gpart, float *dA, float *dW, float *dh, hipStream_t st);

// training step: MSE partial sums (t > T_w), MAR loss and gradient, the loss, one Adam step
size_t train_partials();
int launch_mse_loss_partial(const float *z, const float *x, int B, int T, int M, int N, int T_w, double *part,
                            hipStream_t st);
int launch_mar(bool shallow, const float *A, const float *W, const float *V, const float *h, int M, int L, int M_r,
               float lam, int p, float gw, float gv, float *g, double *mar, hipStream_t st);
int launch_loss_final(const double *part, double scale, const double *mar, float *loss, hipStream_t st);
int launch_adam(float *const *params, const long *sizes, const float *g, float *m, float *v, float lr, float b1,
                float b2, float eps, int step, hipStream_t st);

// quasi-DEER, vanilla PLRNN (diagonal Jacobians): chunk length, one forward Newton update
// (r and gamma d at the current iterate, chunked diagonal scan, z + Delta to the other buffer,
// per-chain maxima), and the quasi adjoint with per-chain gradient partials
// gpart[chain][MP][MP + 2] (MP = padded_dim(M)) for launch_reduce_gpart
int qdeer_chunk_len(int B, int T, int M);
int launch_qdeer_update(const PlrnnArgs &a, float *z, float *zalt, const int *zsel, const int *active,
                        const float *gamma, float *rhs, float *coef, float *P, float *v, float *carry,
                        uint32_t *chain_bits, int C, int ncs, hipStream_t st);
// Fused quasi-DEER passes of the adaptive loop (vanilla PLRNN): one kernel per pass takes the
// fix-up of the previous update, where fc.nd.pv says the aggregates in (Pin, vin, gin) belong to
// the current iterate, and the chunk aggregates of the next update, written to (Pout, vout,
// gout), with the pass-end control.  ncs is a multiple of qdeer_pass_group(M), at most
// qdeer_pass_max_chunks(M) (padding chunks past T are empty).  Block 0 writes pass_no to *mark as it starts.
int qdeer_pass_group(int M);
int qdeer_pass_max_chunks(int M);
int launch_qdeer_pass(const PlrnnArgs &a, float *z, float *zalt, const float *Pin, const float *vin, const double *gin,
                      float *Pout, float *vout, double *gout, int C, int ncs, const FusedCtl &fc, uint32_t *mark,
                      uint32_t pass_no, hipStream_t st);
int launch_qdeer_adjoint(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, float *coef, float *P,
                         float *v, float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st);
// the model-independent parts: the forward scan + fix-up from (rhs = r, coef), and the reverse
// scan from coef (gpart null: no vanilla gradient partials, lam written); shallow-PLRNN
// coefficients from the hidden-unit masks (M L <= 8192)
int launch_qdeer_scan_fwd(int B, int T, int M, const float *x, int N, float *z, float *zalt, const int *zsel,
                          const int *active, const float *rhs, const float *coef, float *P, float *v, float *carry,
                          uint32_t *chain_bits, int C, int ncs, hipStream_t st);
int launch_qdeer_scan_rev(const PlrnnArgs &a, const float *g, float seed_scale, const float *z, const float *coef,
                          float *P, float *v, float *carry, float *lam, float *gpart, int C, int ncs, hipStream_t st);
int launch_qdeer_shdiag(const ShArgs &a, const uint32_t *masks, const int *active, const float *gamma, float *coef,
                        hipStream_t st);

// dense stored-Jacobian scan (mode: 0 Newton fix-up, 1 bare forward scan, 2 reverse)
// flip (bare scan only): the other orientation of every stored matrix than the direction's default
// (forward J_t^T, reverse J_{t+1})
int launch_chunk_product_dense(bool rev, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                               float *P, float *v, const int *active, int C, int ncs, hipStream_t st,
                               bool flip = false);
int launch_fixup_dense(int mode, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                       const float *carry_in, float *z, float *out, const int *zsel, uint32_t *chain_bits,
                       const int *active, int C, int ncs, hipStream_t st, bool flip = false);

// latent dimensions 65..128 (padded width 128; k_big.hip), dispatched to by the launchers above
// and below; the carry takes one level, or two when G > 0 (groups of G chunks, gws as sized by
// carry_ws_floats)
int launch_chunk_product_big(bool rev, bool flip, int B, int T, int M, const float *J, const float *rhs,
                             float rhs_sign, float *P, float *v, const int *active, int C, int ncs, hipStream_t st);
int launch_carry_big(bool rev, const float *P, const float *v, float *carry_in, const int *active, int B, int ncs,
                     int G, float *gws, hipStream_t st);
int launch_fixup_big(int mode, bool flip, int B, int T, int M, const float *J, const float *rhs, float rhs_sign,
                     const float *carry_in, float *z, float *out, const int *zsel, uint32_t *chain_bits,
                     const int *active, int C, int ncs, hipStream_t st);
size_t big_resjac_lds(int M, int L);
size_t big_jacform_lds(int L);
size_t big_grads_lds(int M, int L);
int launch_resjac_big(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *F, float *r,
                      uint32_t *masks, const int *active, hipStream_t st);
int launch_jacform_big(const ShArgs &a, const uint32_t *masks, float *J, const int *active, const float *gamma,
                       hipStream_t st);
int launch_grads_big(const ShArgs &a, const float *z, const float *lam, const uint32_t *masks, float *part, int nb,
                     hipStream_t st);

// shallow PLRNN
// shallow PLRNN Newton update without a stored Jacobian (masks + W1, W2 only)
bool shfused_supported(int M, int L);
size_t shfused_product_lds(int M, int L);
// mark: with the adaptive loop's one-pass-ahead queueing, block 0 writes pass_no to it as it starts
int launch_resjac_shmfma(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *r,
                         uint32_t *masks, const int *active, hipStream_t st, uint32_t *mark = nullptr,
                         uint32_t pass_no = 0u);
// rev: the adjoint's reverse recursion (gamma and active must be null; the fix-up writes y to out)
int launch_chunk_product_shfused(bool rev, const ShArgs &a, const uint32_t *masks, const float *rhs,
                                 float rhs_sign, const float *gamma, float *P, float *v, const int *active, int C,
                                 int ncs, hipStream_t st);
// fc (forward, adaptive loop only): the fix-up takes the pass-end control itself (no chain_bits)
int launch_fixup_shjvp(bool rev, const ShArgs &a, const uint32_t *masks, const float *rhs, float rhs_sign,
                       const float *gamma, const float *carry_in, float *z, float *out, const int *zsel,
                       uint32_t *chain_bits, const int *active, int C, int ncs, hipStream_t st,
                       const FusedCtl *fc = nullptr);
size_t sh_resjac_lds(int M, int L);
size_t sh_jacform_lds(int M, int L);
size_t sh_grads_part_floats(int M, int L, int *nblocks);
int launch_resjac_shplrnn(const ShArgs &a, const float *z, const float *zalt, const int *zsel, float *F, float *r,
                          uint32_t *masks, const int *active, hipStream_t st);
int launch_jacform_shplrnn(const ShArgs &a, const uint32_t *masks, float *J, const int *active, const float *gamma,
                           hipStream_t st);
int launch_grads_shplrnn(const ShArgs &a, const float *z, const float *lam, const uint32_t *masks, float *part,
                         const deer_grads *gr, hipStream_t st);
// rows s < tw (the latent warm-up's states) get no seed
int launch_mse_seed(const float *z, const float *x, float scale, int B, int T, int M, int N, float *g, hipStream_t st,
                    int tw = 0);

// read-out MLP of the diagonal SSM
struct RoArgs {
    const float *Wa, *ca, *Wb, *cb;
    int M, H, No;
};
struct RoGrads {
    float *Wa, *ca, *Wb, *cb;
};
size_t readout_ws_bytes(int B, int T);
int launch_readout(const RoArgs &ra, int B, int T, const float *h, const float *x, float *g, uint32_t *masks,
                   float *loss, const RoGrads &gr, void *ws, hipStream_t st);

// diagonal complex scan
size_t diag_scan_ws_bytes(int B, int T, int M);
// conj < 0: the recursion multiplies by conj(lambda) when rev (the adjoint), else by lambda;
// conj >= 0 chooses conj(lambda) (1) or lambda (0) in either direction
int launch_diag_scan(bool rev, int B, int T, int M, const float *lam, const float *b, const float *Bc, int K,
                     const float *u, float *y, void *ws, hipStream_t st, int conj = -1);
size_t diag_adjoint_ws_bytes(int B, int T, int M, int K);
int launch_diag_adjoint(int B, int T, int M, int K, const float *lam, const float *g, bool g_real, const float *h,
                        const float *x, float *lam_out, float *dlam, float *dBc, void *ws, hipStream_t st);

// sequential baseline (k_seq.hip): one workgroup per sequence, the steps in order
struct SeqArgs {
    const float *A, *W1, *W2, *h1, *h2;   // vanilla: W1 = W (M x M), W2 = h2 = null, L = M
    float alpha;
    int N;
    const float *x, *z0;
    int B, T, M, L;
    bool sh;
};
int seq_check(int M, int L, bool sh);
size_t seq_part_floats(int M, int L, bool sh);
int launch_seq_forward(const SeqArgs &a, float *z, float *act, hipStream_t st);
int launch_seq_backward(const SeqArgs &a, const float *z, const float *act, const float *g, float seed_scale,
                        float *lam, float *part, const deer_grads *gr, hipStream_t st);

// general observation matrix B [N, M] (k_obs.hip)
struct ObsSetup {
    const float *B;          // [N, M]
    int N, M, L;             // L = hidden width (shallow) or M (vanilla, W2 = I)
    float alpha;
    const float *A, *W2;     // W2 null: the identity (vanilla PLRNN)
    double *Bp64, *B64, *P164;                       // B^+ [M, N], B [N, M], P_1 [M, M]
    float *Bp32, *Pa32, *P132, *Ca, *C1, *Id;        // B^+, P_alpha, P_1, diag(A) P_alpha, diag(A) P_1, I
    float *Va, *V1;                                  // W2 P_alpha, W2 P_1 [L, M]
    double *aug;                                     // [64][128] Gauss-Jordan scratch
};
int launch_obs_setup(const ObsSetup &s, hipStream_t st);
// mode 0: forced inputs out[b, s] = P_s z_{s-1} + alpha_s B^+ x_s (s >= 1) of the current iterate;
// mode 1: teacher states out[b, s] = B^+ x_{s+1}.  Both write z0e = B^+ x_0 when z0 is null.
int launch_obs_forced(int mode, const float *z, const float *zalt, const int *zsel, const float *x, const float *z0,
                      const float *Bp, const float *Pa, const float *P1, float alpha, int T_w, int B, int T, int M,
                      int N, float *out, float *z0e, hipStream_t st);
int launch_obs_seed(const float *z, const float *x, const float *Bm, float scale, int T_w, int B, int T, int M, int N,
                    float *g, hipStream_t st);
size_t obs_bgrad_ws_doubles(int M, int N);
int launch_obs_bgrad(const float *JF, const float *lam, const float *z, const float *x, const float *Bm32,
                     const double *Bp64, const double *Bm64, const double *P164, bool z0_given, float alpha, int T_w,
                     bool with_mse, double mse_scale, int B, int T, int M, int N, double *ws, float *gB,
                     hipStream_t st);

// small utilities
int launch_fill_teacher(int B, int T, int M, int N, const float *x, float *z, hipStream_t st);
int launch_fill_i32(int *p, int n, int v, hipStream_t st);
int launch_fill_f32(float *p, size_t n, float v, hipStream_t st);

}  // namespace deer
