/*
 * Fixed-step classical RK4 integrators for the synthetic input trajectories
 * (Lorenz-63 and Lorenz-96, the ODE families of the paper's datasets
 * appendix).  Data generation only: nothing here is part of the DEER method.
 *
 * Built with -ffp-contract=off so that the arithmetic order is exactly the
 * one written below on every host.
 */
#include <stddef.h>

static void l63_rhs(const double *s, double *d, double sigma, double rho, double beta) {
    d[0] = sigma * (s[1] - s[0]);
    d[1] = s[0] * (rho - s[2]) - s[1];
    d[2] = s[0] * s[1] - beta * s[2];
}

/* Integrate n_transient + n_keep steps from state[3]; write the n_keep kept
 * states (row-major [n_keep][3]) to out.  state is updated in place. */
void lorenz63_rk4(double *state, double dt, long n_transient, long n_keep,
                  double sigma, double rho, double beta, double *out) {
    double k1[3], k2[3], k3[3], k4[3], tmp[3];
    long total = n_transient + n_keep;
    for (long step = 0; step < total; ++step) {
        if (step >= n_transient) {
            double *o = out + 3 * (step - n_transient);
            o[0] = state[0]; o[1] = state[1]; o[2] = state[2];
        }
        l63_rhs(state, k1, sigma, rho, beta);
        for (int i = 0; i < 3; ++i) tmp[i] = state[i] + 0.5 * dt * k1[i];
        l63_rhs(tmp, k2, sigma, rho, beta);
        for (int i = 0; i < 3; ++i) tmp[i] = state[i] + 0.5 * dt * k2[i];
        l63_rhs(tmp, k3, sigma, rho, beta);
        for (int i = 0; i < 3; ++i) tmp[i] = state[i] + dt * k3[i];
        l63_rhs(tmp, k4, sigma, rho, beta);
        for (int i = 0; i < 3; ++i)
            state[i] += dt / 6.0 * (k1[i] + 2.0 * k2[i] + 2.0 * k3[i] + k4[i]);
    }
}

static void l96_rhs(const double *s, double *d, long n, double forcing) {
    /* interior indices without modulo; the three wrapped ones explicitly */
    for (long i = 2; i < n - 1; ++i)
        d[i] = (s[i + 1] - s[i - 2]) * s[i - 1] - s[i] + forcing;
    d[0] = (s[1] - s[n - 2]) * s[n - 1] - s[0] + forcing;
    d[1] = (s[2] - s[n - 1]) * s[0] - s[1] + forcing;
    d[n - 1] = (s[0] - s[n - 3]) * s[n - 2] - s[n - 1] + forcing;
}

/* Same contract as lorenz63_rk4 for the n-dimensional Lorenz-96 system with
 * cyclic indices; work must hold 5*n doubles. */
void lorenz96_rk4(double *state, long n, double dt, long n_transient, long n_keep,
                  double forcing, double *work, double *out) {
    double *k1 = work, *k2 = work + n, *k3 = work + 2 * n, *k4 = work + 3 * n, *tmp = work + 4 * n;
    long total = n_transient + n_keep;
    for (long step = 0; step < total; ++step) {
        if (step >= n_transient) {
            double *o = out + n * (step - n_transient);
            for (long i = 0; i < n; ++i) o[i] = state[i];
        }
        l96_rhs(state, k1, n, forcing);
        for (long i = 0; i < n; ++i) tmp[i] = state[i] + 0.5 * dt * k1[i];
        l96_rhs(tmp, k2, n, forcing);
        for (long i = 0; i < n; ++i) tmp[i] = state[i] + 0.5 * dt * k2[i];
        l96_rhs(tmp, k3, n, forcing);
        for (long i = 0; i < n; ++i) tmp[i] = state[i] + dt * k3[i];
        l96_rhs(tmp, k4, n, forcing);
        for (long i = 0; i < n; ++i)
            state[i] += dt / 6.0 * (k1[i] + 2.0 * k2[i] + 2.0 * k3[i] + k4[i]);
    }
}
