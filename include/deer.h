/*
 * deer.h - C ABI of libdeer: the GTF-DEER hot path on AMD Instinct MI355X (gfx950).
 *
 * GTF-DEER (Hess, Goetz, Durstewitz, "Parallel-in-Time Training of Recurrent
 * Neural Networks for Dynamical Systems Reconstruction") solves the forced
 * recurrence z_t = F(z~_{t-1}) for all t at once by Newton's method: every
 * iteration evaluates the residual and the forced Jacobians at all steps and
 * solves the linear recursion Delta_t = J~_t Delta_{t-1} - r_t with a parallel
 * associative scan (section "DSR from long sequences", eqs. GTF_residual and
 * GTF_DEER_update; Alg. GTF-DEER).  Gradients come from the implicit function
 * theorem: one scan of the same kind, run backwards with transposed Jacobians
 * (gradients appendix, eqs. adjoint_eq and backward_recursion).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All arrays are float32, row-major, contiguous, batch-major and live in
 *    device memory, except where an argument is marked "host".
 *  - x    [B, T+1, N]  observations x_0..x_T (N = forcing.n_forced).
 *  - z    [B, T, M]    states z_1..z_T; z[b, k] is z_{k+1}.
 *  - z0   [B, M]       initial state; NULL means z_0 = B^+ x_0 = [x_0; 0].
 *  - Observation model B = [I_N 0] (identity read-out of the first N latents,
 *    model-setup appendix), so P_alpha = I - alpha B^+ B = diag(1 - a) with
 *    a_i = alpha for i < N and a_i = 0 otherwise (eq. error_forcing).
 *  - Step k+1 (array index k) reads the forced state
 *        z~_k = (1 - a) * z_k + a * [x_k; 0]   for k >= 1,   z~_0 = z_0,
 *    computed in float32 as fl(fl(p*z) + fl(a*zbar)), p = fl(1 - a), no fused
 *    multiply-add, so that the ReLU decision below is reproducible bit for bit.
 *  - masks [B, T, W] uint32, W = ceil(H/32): bit j of step k is (u_j > 0) with
 *    u = z~_k (vanilla PLRNN, H = M) or u = h2 + W2 z~_k (shallow PLRNN, H = L;
 *    u accumulated left to right in j from h2 in float32, one rounding after
 *    every multiply and every add).  phi'(0) = 0.
 *  - Every call runs on `stream` (a hipStream_t; NULL = the null stream).
 *    Buffers are owned by the caller; the library never allocates or frees
 *    device memory.  Scratch space comes from `ws` (device, `ws_bytes` bytes,
 *    at least deer_workspace_bytes(...); 256-byte aligned).
 *  - Errors are returned as a status code (never thrown across the ABI);
 *    argument errors are detected before any device work is queued.
 *    deer_last_error() gives a thread-local message for the last failure.
 *  - Process-wide state (nothing else is kept between calls):
 *      * one pinned host block per host thread, through which the device reports
 *        stopped sequences to the Newton loop of a solve with a tolerance; it is
 *        allocated only by deer_host_reserve and freed by deer_host_release, never
 *        inside a solve;
 *      * the timing diagnostics (deer_timing_*), off unless enabled, which keep a
 *        mutex-protected pool of HIP events;
 *      * the read-out's resident-block count (an occupancy query made once per
 *        process) and, per GPU, the scratch array of deer_scan_noalloc.
 *    Calls on different streams with different workspaces may run concurrently;
 *    calls that share a workspace must be serialised by the caller, and one host
 *    thread runs its solves one at a time.
 */
#ifndef DEER_H
#define DEER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------------- */
enum {
    DEER_OK = 0,
    DEER_ERR_INVALID_ARG = 1,     /* null pointer, B/T/M out of range, alpha not in [0,1], ... */
    DEER_ERR_NOT_CONVERGED = 2,   /* max_iter reached; z holds the last iterate */
    DEER_ERR_NONFINITE = 3,       /* a Newton update produced NaN or Inf */
    DEER_ERR_HIP = 4,             /* a HIP runtime call failed */
    DEER_ERR_WORKSPACE = 5        /* ws too small or misaligned */
};

/* ---- models ------------------------------------------------------------------------ */
enum {
    DEER_PLRNN = 0,    /* z' = diag(A) z~ + W relu(z~) + h                       (W [M,M])   */
    DEER_SHPLRNN = 1,  /* z' = diag(A) z~ + W relu(W2 z~ + h2) + h     (W [M,L], W2 [L,M])  */
    DEER_DIAG_SSM = 2  /* h' = lambda * h + Bc u (complex diagonal, eq. shplrnn_ssm)        */
};

/* Parameters (device pointers).  The PLRNN kinds are eq. shplrnn_nonlinear with
 * V = I, b = 0 (vanilla) or V = W2, b = h2 (shallow); no external inputs.
 * DEER_DIAG_SSM: A = lambda [M][2] (re, im), W = Bc [M, L][2] with L the input
 * dimension (inputs u_t = x_{t-1}), other pointers unused. */
typedef struct {
    int kind;
    int M;              /* latent dimension: 1..64 for the vanilla PLRNN, 1..128 for the shallow
                           one (M > 64: L <= 62, M L <= 7936; quasi-DEER and an observation
                           matrix up to 64), >= 1 for DIAG_SSM */
    int L;              /* shallow: hidden width (1..1024); DIAG_SSM: input dimension       */
    const float *A;
    const float *W;
    const float *W2;
    const float *h;     /* may be NULL (zero) */
    const float *h2;    /* may be NULL (zero) */
} deer_model;

typedef struct {
    float alpha;        /* GTF forcing strength in [0, 1] (eq. GTF)                          */
    int n_forced;       /* N: the first N latents are observed and forced, 0 <= N <= M      */
    int T_w;            /* latent warm-up (Alg. GTF-DEER, latent state warm-up paragraph):
                           0 <= T_w < T; the forced inputs z~_1..z~_{T_w} use alpha = 1 and
                           the MSE seed leaves z_1..z_{T_w} out (1 / (N (T - T_w))).  PLRNN
                           kinds; the workspace is deer_workspace_bytes_ex(...).            */
    const float *obs;   /* general observation matrix B [n_forced, M] (device, row-major) of the
                           read-out x^_t = B z_t, or NULL for the identity read-out B = [I_N 0].
                           With B given (PLRNN kinds, 1 <= n_forced <= 64, n_forced may exceed
                           M; B of full rank min(N, M)): the forcing of eq. error_forcing with
                           the dense projector P_alpha = I - alpha B^+ B and targets B^+ x_t,
                           J~_t = J_F(z~_{t-1}) P_alpha (eq. error_forcing_decomp), z_0 = B^+ x_0
                           and the initial iterate B^+ x_{1:T}; the MSE seed is 2/(B N (T - T_w))
                           B^T (B z_t - x_t); a warm-up (T_w > 0) uses P_1 = I - B^+ B and alpha = 1
                           for z~_1..z~_{T_w} inside the same Newton iteration (Alg. GTF-DEER).
                           B^+ and the projectors are formed on the device at the start of each
                           call; a rank-deficient B makes them NaN (the solve then returns
                           DEER_ERR_NONFINITE).  Supported by deer_solve and deer_adjoint(_ex);
                           the other entry points return DEER_ERR_INVALID_ARG for it.           */
} deer_forcing;

enum { DEER_INIT_TEACHER = 0, DEER_INIT_ZERO = 1, DEER_INIT_USER = 2 };

typedef struct {
    float tol;          /* stop a sequence once max_{t,m} |Delta z| < tol (absolute)        */
    int max_iter;       /* cap on Newton passes (accepted or rejected, 500 if <= 0)         */
    int fixed_iters;    /* > 0: run exactly this many updates, no convergence test/sync     */
    int init;           /* DEER_INIT_*: z^(0) = [x_{1:T}; 0], zeros, or z as passed in       */
    float step_bound;   /* rejection threshold (see deer_solve); 0: 1e3; < 0: reject only
                           non-finite updates                                               */
} deer_solve_opts;

/* Per-parameter gradient outputs (device, float32, NULL to skip).
 * PLRNN: A [M], W [M,M], h [M].  SHPLRNN: A [M], W [M,L] (=W1), W2 [L,M], h [M] (=h1),
 * h2 [L].  DIAG_SSM: A = dlambda [M][2], W = dBc [M,L][2] (d/dRe + i d/dIm).
 * obs [N,M]: dL/dB when the forcing has an observation matrix B (Alg. GTF-DEER, g_B): the
 * dependence of the forced inputs, of z_0 = B^+ x_0 and of the MSE on B.  With a cotangent g
 * given instead of the MSE seed, only the first two (sum_t lam_t^T dF(z~_{t-1})/dB). */
typedef struct {
    float *A;
    float *W;
    float *W2;
    float *h;
    float *h2;
    float *obs;
} deer_grads;

enum { DEER_OP_SOLVE = 0, DEER_OP_ADJOINT = 1, DEER_OP_JACOBIAN = 2 /* plrnn_jacobian_ex */ };
enum { DEER_SCAN_DENSE = 0, DEER_SCAN_DIAG_C64 = 1 };

/* Bytes of workspace `op` (DEER_OP_SOLVE or DEER_OP_ADJOINT) needs for this model and
 * size (no warm-up).  Returns 0 for invalid arguments. */
size_t deer_workspace_bytes(const deer_model *model, int B, int T, int op);

/* The same for any forcing, warm-up included, and for the quasi-DEER entry points when
 * quasi != 0.  A latent warm-up (T_w > 0) is part of the one Newton iteration (Alg. GTF-DEER:
 * the kernels take alpha_s = 1 and P_1 for s <= T_w; quasi-DEER the same in its diagonal
 * coefficients), so iters and fixed_iters count updates of the whole sequence and, with the
 * identity read-out, the workspace is that of the plain solve.  With an observation matrix
 * (forcing->obs) the workspace holds the projectors and the stored Jacobians. */
size_t deer_workspace_bytes_ex(const deer_model *model, const deer_forcing *forcing, int B, int T, int op,
                               int quasi);

/* GTF-DEER forward solve (Alg. GTF-DEER, Newton loop; eqs. GTF_residual, GTF_DEER_update).
 *   x, z0        inputs as above; z0 may be NULL.
 *   z            [B,T,M] out (in as well when opts->init == DEER_INIT_USER).  For
 *                DEER_DIAG_SSM, z is h [B,T,M][2] (complex) and the call is the single
 *                linear scan h_t = lambda h_{t-1} + Bc x_{t-1}, h_0 = 0 (Alg. LSSM).
 *   masks        [B,T,W] out or NULL: activation masks at the returned z.
 *   iters        host [B] out or NULL: updates applied (accepted) to each sequence,
 *                counting the verifying one (a sequence converged after k updates reports k).
 *   final_norm   host [B] out or NULL: max |Delta z| of each sequence's last update.
 * Each Newton update is applied before the test; a sequence whose update is below tol
 * is frozen while the others continue.  With fixed_iters == 0 the test runs on the device
 * after every update; a sequence that stops clears a flag in the calling thread's pinned host
 * block (deer_host_reserve(B) must have been called on this thread; otherwise the call returns
 * DEER_ERR_INVALID_ARG before any device work), which also receives its update count, last
 * norm and status.  The host keeps passes queued ahead
 * of the device and returns once every sequence has stopped (then without a stream
 * synchronisation: z is complete in stream order, and the passes still queued skip every
 * sequence) or at max_iter (after a synchronisation).  Calls from one host thread run one
 * at a time.  The loop also safeguards the
 * iteration: an update that is not finite, or whose max|Delta z| exceeds
 * step_bound * (1 + max|z|) of its sequence, is discarded and that sequence retried with
 * the damped linearisation gamma J~ (0 <= gamma < 1; gamma = 0 is the fixed-point step
 * z_t = F(z~_{t-1})), gamma returning to 1 (plain Newton) over accepted updates.  Every
 * gamma has the same fixed point and the same prefix property (one more leading step exact
 * per update), so the solution is unchanged; only the path to it differs.  With
 * fixed_iters > 0 the updates are plain Newton steps applied unconditionally and the call
 * synchronises once at the end (to read the final norms).
 * Returns DEER_OK, DEER_ERR_NOT_CONVERGED (z = last accepted iterate), DEER_ERR_NONFINITE
 * (also when the undamped fixed-point step overflows) or an argument / HIP / workspace
 * error. */
int deer_solve(const deer_model *model, const deer_forcing *forcing, const deer_solve_opts *opts,
               int B, int T, const float *x, const float *z0, float *z, uint32_t *masks,
               int32_t *iters, float *final_norm, void *ws, size_t ws_bytes, void *stream);

/* Adjoint of the forced recurrence at a (converged) trajectory z (gradients appendix):
 *   lam_T = g_T,  lam_{t-1} = J~_t^T lam_t + g_{t-1},   J~_t = J_F(z~_{t-1}) P_alpha,
 * i.e. lam = dL/dz (the paper's v with the opposite sign), and the parameter gradients
 *   dL/dtheta = sum_{b,t} lam_t^T dF(z~_{t-1})/dtheta.
 *   g     [B,T,M] or NULL.  NULL: the MSE seed g_t = 2/(B N T) [z_t[:N] - x_t; 0] of the
 *         batch-mean loss (eq. mse_loss_series).  DIAG_SSM: g is required, complex
 *         [B,T,M][2] = dL/dRe h + i dL/dIm h, the recursion uses conj(lambda), and z is
 *         the forward h.
 *   lam   [B,T,M] out (DIAG_SSM: [B,T,M][2]) or NULL.
 *   grads per-parameter outputs or NULL (sums over all (b, t), reduced in float64).
 * Fully asynchronous on `stream`. */
int deer_adjoint(const deer_model *model, const deer_forcing *forcing, int B, int T,
                 const float *x, const float *z0, const float *z, const float *g,
                 float *lam, const deer_grads *grads, void *ws, size_t ws_bytes, void *stream);

/* Quasi-DEER (PLRNN kinds): deer_solve and deer_adjoint with every forced Jacobian
 * J~_t replaced by its diagonal d_t = diag(J_F(z~_{t-1})) P_alpha, i.e.
 * d_t[i] = (A_i + W_ii 1[z~_{t-1,i} > 0]) (1 - a_i) for the vanilla PLRNN and
 * d_t[i] = (A_i + sum_l W_il 1[u_l > 0] W2_li) (1 - a_i), u = W2 z~_{t-1} + h2, for the shallow
 * one (same limits as deer_solve) -- the quasi-Newton variant the paper sets
 * against full Jacobians (section on DEER, the diagonal approximation of eq. DEER_update;
 * quasi form of the backward recursion in the gradients appendix; ablation of Jacobian
 * diagonalisation).  Updates: Delta_t = d_t Delta_{t-1} - r_t (the same zero of the residual,
 * so a converged solve equals deer_solve's, usually after many more updates).  Adjoint:
 * lam_T = g_T, lam_{t-1} = d_t lam_t + g_{t-1}, gradients sum lam_t^T dF(z~_{t-1})/dtheta
 * as in deer_adjoint (an approximation of the true gradient that ignores the mixing between
 * latents).  Arguments, outputs, the safeguard and the status codes are those of
 * deer_solve / deer_adjoint; the workspace is deer_quasi_workspace_bytes(model, B, T, op)
 * bytes.  DEER_DIAG_SSM returns DEER_ERR_INVALID_ARG (its recurrence is already diagonal). */
int deer_solve_quasi(const deer_model *model, const deer_forcing *forcing, const deer_solve_opts *opts,
                     int B, int T, const float *x, const float *z0, float *z, uint32_t *masks,
                     int32_t *iters, float *final_norm, void *ws, size_t ws_bytes, void *stream);
int deer_adjoint_quasi(const deer_model *model, const deer_forcing *forcing, int B, int T,
                       const float *x, const float *z0, const float *z, const float *g,
                       float *lam, const deer_grads *grads, void *ws, size_t ws_bytes, void *stream);
size_t deer_quasi_workspace_bytes(const deer_model *model, int B, int T, int op);

/* Hyper-parameters of deer_train_step. */
typedef struct {
    float lr, beta1, beta2, eps;   /* Adam (the paper names no optimiser; Adam is the reading)   */
    int step;                      /* Adam step t >= 1 (bias corrections 1 - beta^t)             */
    float mar_lambda;              /* MAR weight lambda_MAR (0: no MAR term)                      */
    int mar_units;                 /* M_r: MAR acts on the last M_r latents, 1 <= M_r <= M       */
    int mar_p;                     /* 1 or 2: |.| or squared penalty                             */
    float mar_gamma_w, mar_gamma_v;/* scales of the W and V terms (the paper: 1/(3L), 1/(3M))    */
    int quasi;                     /* quasi-DEER solve and adjoint instead of GTF-DEER           */
} deer_train_opts;

/* One training step of GTF-DEER (Alg. GTF-DEER, the body of its outer loop), PLRNN kinds:
 *   the solve to opts->tol (deer_solve, or deer_solve_quasi), the loss
 *     L = MSE(x_{T_w+1:T}, B z_{T_w+1:T}) + L_MAR (eqs. mse_loss_warmup, mar_loss_latent_initscale;
 *     L_MAR = lambda/M_r sum_{i > M - M_r} [|1 - A_i|^p + (1/L) sum_j (gamma_W |W_ij|^p
 *     + gamma_V |V_ji|^p) + |h_i|^p], V = W2 and W = W1 for the shallow model, no V term and
 *     L = M for the vanilla one),
 *   its gradient (deer_adjoint with the MSE seed, plus the MAR gradient), and one Adam step
 *   applied IN PLACE to the parameter arrays the model points at (A, W, W2, h, h2; a NULL h or
 *   h2 stays NULL and untrained).
 *   z          [B,T,M] out: the solved trajectory (the iterate the gradient is taken at).
 *   adam_m/v   [P] device, in/out: Adam moments in the layout A | W | h (vanilla) or
 *              A | W1 | W2 | h1 | h2 (shallow), P = deer_train_params(model); zero before step 1.
 *   grads      optional outputs of the total gradient (MSE + MAR) before the update, or NULL.
 *   loss       device [1] out or NULL;  iters host [B] out or NULL.
 * If the solve does not converge (or is non-finite) its status is returned and the
 * parameters are left unchanged.  Workspace: deer_train_workspace_bytes(model, forcing, B, T,
 * train->quasi). */
int deer_train_step(const deer_model *model, const deer_forcing *forcing, const deer_solve_opts *opts,
                    const deer_train_opts *train, int B, int T, const float *x, const float *z0, float *z,
                    float *adam_m, float *adam_v, const deer_grads *grads, float *loss, int32_t *iters,
                    void *ws, size_t ws_bytes, void *stream);
size_t deer_train_workspace_bytes(const deer_model *model, const deer_forcing *forcing, int B, int T, int quasi);
size_t deer_train_params(const deer_model *model);

/* Sequential GTF baseline (the comparison of Fig. 1A): the forward rollout
 *   z_s = F(z~_s), z~ the forced state of eq. GTF, step by step in time,
 * and, when lam or grads is given, back-propagation through time, also step by step:
 *   lam_{T-1} = g_{T-1},  lam_s = g_s + J~_{s+1}^T lam_{s+1},  dL/dtheta = sum lam_s^T dF/dtheta.
 * The outputs are those of deer_solve at convergence and deer_adjoint at its z, computed in
 * time order with the batch as the only parallel dimension (one workgroup per sequence):
 * the training the parallel solver replaces.  PLRNN kinds only; M <= 256, L <= 256,
 * M L <= 8192 (vanilla: M^2 <= 8192), and the weights must fit in 160 KiB of LDS.
 *   x, z0        as in deer_solve;  z [B,T,M] out.
 *   g            [B,T,M] or NULL (the MSE seed, as in deer_adjoint).
 *   lam          [B,T,M] out or NULL;  grads as in deer_adjoint or NULL (then no backward pass
 *                when lam is NULL too).
 *   ws           deer_sequential_workspace_bytes(model, B, T) bytes.
 * Fully asynchronous on `stream`. */
int deer_sequential(const deer_model *model, const deer_forcing *forcing, int B, int T,
                    const float *x, const float *z0, float *z, const float *g, float *lam,
                    const deer_grads *grads, void *ws, size_t ws_bytes, void *stream);
size_t deer_sequential_workspace_bytes(const deer_model *model, int B, int T);

/* Layout of the cotangent g of deer_adjoint_ex. */
enum { DEER_G_NATIVE = 0, DEER_G_REAL = 1 };

/* deer_adjoint with an explicit cotangent layout.  DEER_G_NATIVE is deer_adjoint.
 * DEER_G_REAL (DEER_DIAG_SSM only): g is [B,T,M] real, dL/dRe h with dL/dIm h = 0 -- the
 * cotangent the read-out MLP supplies (deer_readout_loss), read at 4 bytes per element. */
int deer_adjoint_ex(const deer_model *model, const deer_forcing *forcing, int B, int T,
                    const float *x, const float *z0, const float *z, const float *g, int g_layout,
                    float *lam, const deer_grads *grads, void *ws, size_t ws_bytes, void *stream);

/* Read-out MLP of the diagonal SSM and its loss (linear-SSM appendix: the LSSM's
 * observation model; the MSE of eq. mse_loss_series on its outputs):
 *   s_t = Wa Re(h_t) + ca,  y_t = Wb relu(s_t) + cb,
 *   L = sum_{b,t} ||y_t - x_t||^2 / (B No T), with h_t the state after input x_{t-1}
 *       (0-based arrays: state row t is compared with x row t + 1).
 * Sizes: M <= 64 state channels, H <= 128 hidden units, No <= 4 outputs (= input dim K). */
typedef struct {
    int H;              /* hidden units                                                     */
    int n_out;          /* No: outputs, equal to the data dimension of x                    */
    const float *Wa;    /* [H, M]                                                           */
    const float *ca;    /* [H] or NULL (zero)                                               */
    const float *Wb;    /* [No, H]                                                          */
    const float *cb;    /* [No] or NULL (zero)                                              */
} deer_readout;

typedef struct {
    float *Wa, *ca, *Wb, *cb;   /* gradient outputs (device, same shapes) or NULL to skip    */
} deer_readout_grads;

/* Workspace bytes deer_readout_loss needs. */
size_t deer_readout_workspace_bytes(const deer_readout *readout, int B, int T, int M);

/* Forward and backward pass of the read-out at the states h [B,T,M][2] (complex):
 *   g     [B,T,M] out (required): dL/dRe h_t = Wa^T ((Wb^T dy_t) * 1[s_t > 0]),
 *         dy_t = 2 (y_t - x_{t+1}) / (B No T); feed it to deer_adjoint_ex(DEER_G_REAL).
 *   loss  device [1] out or NULL.
 *   masks [B,T,ceil(H/32)] out or NULL: the ReLU decisions 1[s_t > 0] taken (bit j of word
 *         w is hidden unit 32 w + j).
 *   grads read-out parameter gradients or NULL (sums over all (b, t), reduced in float64).
 * Fully asynchronous on `stream`. */
int deer_readout_loss(const deer_readout *readout, int B, int T, int M, const float *h, const float *x,
                      float *g, float *loss, uint32_t *masks, const deer_readout_grads *grads, void *ws,
                      size_t ws_bytes, void *stream);

/* Residual and forced Jacobians of a PLRNN kind at trajectory z (eq. GTF_residual; the
 * Jacobian of F in the model-setup appendix; eq. error_forcing_decomp):
 *   F     [B,T,M] out or NULL: F(z~_{t-1}).
 *   r     [B,T,M] out or NULL: z_t - F(z~_{t-1}).
 *   J     [B,T,M,M] out or NULL: J~_t = J_F(z~_{t-1}) P_alpha, row-major per step.
 *   masks [B,T,W] out or NULL.
 * No workspace; fully asynchronous. */
int plrnn_jacobian(const deer_model *model, const deer_forcing *forcing, int B, int T,
                   const float *x, const float *z0, const float *z, float *F, float *r, float *J,
                   uint32_t *masks, void *stream);

/* plrnn_jacobian for any forcing: with forcing->obs (a general observation matrix; a warm-up
 * T_w > 0 allowed) the residual, masks and forced Jacobians of that forcing, computed by the
 * same kernels deer_solve and deer_adjoint use (so the masks are the decisions they take), with
 * deer_workspace_bytes_ex(model, forcing, B, T, DEER_OP_JACOBIAN, 0) bytes of workspace; without
 * obs it is plrnn_jacobian (ws unused).  Fully asynchronous. */
int plrnn_jacobian_ex(const deer_model *model, const deer_forcing *forcing, int B, int T,
                      const float *x, const float *z0, const float *z, float *F, float *r, float *J,
                      uint32_t *masks, void *ws, size_t ws_bytes, void *stream);

/* The bare associative scan over affine pairs (scheduled-sampling appendix: the pair
 * (A_t, b_t) and its composition), batched over B independent sequences of length T.
 * `reverse` chooses the direction, `transpose` whether each step applies its matrix (0) or
 * its transpose (1); the Newton update of eq. GTF_DEER_update is (reverse, transpose) = (0, 0)
 * and the adjoint recursion of eq. backward_recursion is (1, 1).  With op(J) = J or J^T:
 *   DEER_SCAN_DENSE:    J [B,T,M,M] row-major per step, b [B,T,M], M <= 128.
 *        reverse == 0:  y_t = op(J_t) y_{t-1} + b_t, y_0 = 0        (J_1 is not read)
 *        reverse != 0:  y_T = b_T, y_{t-1} = op(J_t) y_t + b_{t-1}  (J_1 is not read)
 *   DEER_SCAN_DIAG_C64: J = lambda [M][2], b [B,T,M][2] complex; op(lambda) = lambda, or
 *        conj(lambda) with transpose != 0 (C read as R^2, where multiplication by lambda is
 *        the 2 x 2 block [[Re, -Im], [Im, Re]] and its transpose is multiplication by conj):
 *        reverse == 0:  y_t = op(lambda) y_{t-1} + b_t, y_0 = 0
 *        reverse != 0:  y_T = b_T, y_{t-1} = op(lambda) y_t + b_{t-1}
 *   y     out, same layout as b (may not alias b).
 * The scan takes explicit matrices; the mask-driven Jacobians of the PLRNN kinds are formed
 * inside deer_solve / deer_adjoint, which know the model.  Fully asynchronous. */
int deer_scan(int layout, int reverse, int transpose, int B, int T, int M, const float *J, const float *b,
              float *y, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes deer_scan needs for these arguments (0 if they are invalid). */
size_t deer_scan_workspace_bytes(int layout, int reverse, int transpose, int B, int T, int M);

/* deer_scan for callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc): the same scan with the same arguments and
 * results, its scratch in a static device array of the library (deer_noalloc_scratch_bytes()
 * = 64 MiB per GPU, held by each GPU the library runs on until the process ends) instead of a
 * workspace.  The call allocates nothing (no hipMalloc, no events: the timing diagnostics skip
 * it).  Sizes whose deer_scan_workspace_bytes exceeds the array are rejected with
 * DEER_ERR_INVALID_ARG before any device work.  Every call on one GPU uses that GPU's array,
 * which keeps the last call's contents: calls that overlap on one GPU (other streams, other
 * threads) race and must be serialised by the caller.  Fully asynchronous on `stream`. */
int deer_scan_noalloc(int layout, int reverse, int transpose, int B, int T, int M, const float *J,
                      const float *b, float *y, void *stream);
size_t deer_noalloc_scratch_bytes(void);

/* Reserves the calling host thread's pinned host block for solves with a tolerance of up to
 * max_batch sequences (deer_solve, deer_solve_quasi, deer_train_step): (4 max_batch + 32)
 * 32-bit words of device-coherent pinned host memory, through which the device reports each
 * sequence that stops (its flag, update count, last norm and status) and the start of each
 * forward pass, so the host follows the Newton loop without copies or stream synchronisation.
 * A block that already holds max_batch sequences is kept (no call); a smaller one is replaced.
 * Call it once per thread at set-up, outside any solve of that thread.  Returns DEER_OK,
 * DEER_ERR_INVALID_ARG (max_batch <= 0) or DEER_ERR_HIP (the pinned allocation failed). */
int deer_host_reserve(int max_batch);

/* Frees the calling thread's pinned host block (no-op without one); a later solve with a
 * tolerance on this thread needs deer_host_reserve again. */
int deer_host_release(void);

/* Diagnostics: per-kernel timing with HIP events.  While enabled, every kernel launch is
 * bracketed by two events recorded on the stream it is launched on (the caller's stream).
 * deer_timing_enable(1) clears earlier records and starts recording; deer_timing_enable(0)
 * stops.  deer_timing_report(idx, ...) waits for the events of the idx-th distinct kernel
 * (in first-launch order) and returns its name, total milliseconds and launch count; the
 * return value is the number of distinct kernels recorded (negative on a HIP error).
 * Process-wide; meant for benchmarks, not for concurrent production calls. */
int deer_timing_enable(int on);
int deer_timing_report(int idx, char *name, int name_cap, double *ms_total, long *launches);

/* Static description of a status code; never NULL. */
const char *deer_status_string(int status);

/* Thread-local message describing the last failing call on this thread ("" if none). */
const char *deer_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DEER_H */
