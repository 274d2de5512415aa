/*
 * swr_oracle.c -- plain double-precision CPU oracle for the Sliding Window
 * Recurrence (test infrastructure only; see swr_oracle.h for the definition,
 * the layouts and who may use this file).
 *
 * Nothing here is blocked, fused or reordered: the forward walks every block's
 * window token by token (the recurrence of Sec. 3, eq. (2.1), restarted from
 * zero state at the start of the previous block, which is what the truncation
 * T ~ I_b of Sec. 4.2 keeps), and the backward walks the same windows in
 * reverse, accumulating the chain rule of that loop.
 */
#include "swr_oracle.h"

#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Decay coefficient of token m, channel mu. */
static double decay(const double* a, int a_per_channel, int64_t D, int64_t m, int64_t mu) {
    return a_per_channel ? a[m * D + mu] : a[m];
}

static int bad_args(int64_t T, int64_t D, int64_t block) {
    return T < 0 || D < 1 || block < 1;
}

int swr_oracle_forward_slice(int64_t T, int64_t D, int64_t block, int a_per_channel,
                             int flags, const double* x, const double* a,
                             const double* b, const double* c, double* y) {
    if (bad_args(T, D, block)) return -1;
    if (T == 0) return 0;
    if (!x || !a || !b || !c || !y) return -1;
    double* s = (double*)malloc((size_t)D * sizeof(double));
    if (!s) return -1;
    const int64_t nblocks = (T + block - 1) / block;
    for (int64_t tau = 0; tau < nblocks; ++tau) {
        /* Window of block tau: the previous block (if any) and block tau itself. */
        const int64_t first = tau * block;
        const int64_t start = (tau > 0 ? tau - 1 : 0) * block;
        const int64_t end = (first + block < T) ? first + block : T;
        for (int64_t mu = 0; mu < D; ++mu) s[mu] = 0.0;
        for (int64_t m = start; m < end; ++m) {
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu;
                s[mu] = decay(a, a_per_channel, D, m, mu) * s[mu] + b[e] * x[e];
                if (m >= first) {
                    y[e] = c[e] * s[mu];
                    if (flags & SWR_ORACLE_RESIDUAL) y[e] += x[e];
                }
            }
        }
    }
    free(s);
    return 0;
}

int swr_oracle_backward_slice(int64_t T, int64_t D, int64_t block, int a_per_channel,
                              int flags, const double* x, const double* a,
                              const double* b, const double* c, const double* dy,
                              double* dx, double* da, double* db, double* dc) {
    if (bad_args(T, D, block)) return -1;
    if (T == 0) return 0;
    if (!x || !a || !b || !c || !dy || !dx || !da || !db || !dc) return -1;
    const int64_t win = 2 * block; /* longest window */
    double* du = (double*)calloc((size_t)(T * D), sizeof(double));
    double* pre = (double*)malloc((size_t)(win * D) * sizeof(double));
    double* post = (double*)malloc((size_t)(win * D) * sizeof(double));
    double* lam = (double*)malloc((size_t)D * sizeof(double));
    if (!du || !pre || !post || !lam) {
        free(du); free(pre); free(post); free(lam);
        return -1;
    }
    memset(da, 0, (size_t)(a_per_channel ? T * D : T) * sizeof(double));

    const int64_t nblocks = (T + block - 1) / block;
    for (int64_t tau = 0; tau < nblocks; ++tau) {
        const int64_t first = tau * block;
        const int64_t start = (tau > 0 ? tau - 1 : 0) * block;
        const int64_t end = (first + block < T) ? first + block : T;
        /* Re-run the window, keeping each step's incoming and outgoing state. */
        for (int64_t mu = 0; mu < D; ++mu) lam[mu] = 0.0; /* lam doubles as the state here */
        for (int64_t m = start; m < end; ++m) {
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu, w = (m - start) * D + mu;
                pre[w] = lam[mu];
                lam[mu] = decay(a, a_per_channel, D, m, mu) * lam[mu] + b[e] * x[e];
                post[w] = lam[mu];
            }
        }
        /* Reverse sweep: lam is d(loss)/d(state after step m). */
        for (int64_t mu = 0; mu < D; ++mu) lam[mu] = 0.0;
        for (int64_t m = end - 1; m >= start; --m) {
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu, w = (m - start) * D + mu;
                if (m >= first) {            /* y_m = c_m * state_m belongs to this window */
                    lam[mu] += c[e] * dy[e];
                    dc[e] = dy[e] * post[w];
                }
                du[e] += lam[mu];            /* d state_m / d u_m = 1          */
                if (a_per_channel)           /* d state_m / d a_m = state_{m-1} */
                    da[e] += lam[mu] * pre[w];
                else
                    da[m] += lam[mu] * pre[w];
                lam[mu] *= decay(a, a_per_channel, D, m, mu); /* d state_m / d state_{m-1} */
            }
        }
    }
    /* u = b * x: chain rule into the two gates; the residual adds dy to dx. */
    for (int64_t e = 0; e < T * D; ++e) {
        dx[e] = b[e] * du[e];
        if (flags & SWR_ORACLE_RESIDUAL) dx[e] += dy[e];
        db[e] = x[e] * du[e];
    }
    free(du); free(pre); free(post); free(lam);
    return 0;
}

int swr_oracle_forward(int64_t S, int64_t T, int64_t D, int64_t block, int a_per_channel,
                       int flags, const double* x, const double* a, const double* b,
                       const double* c, double* y) {
    if (S < 0 || bad_args(T, D, block)) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_forward_slice(T, D, block, a_per_channel, flags, x + s * n, a + s * na,
                                        b + s * n, c + s * n, y + s * n) != 0;
    return err ? -1 : 0;
}

int swr_oracle_backward(int64_t S, int64_t T, int64_t D, int64_t block, int a_per_channel,
                        int flags, const double* x, const double* a, const double* b,
                        const double* c, const double* dy, double* dx, double* da,
                        double* db, double* dc) {
    if (S < 0 || bad_args(T, D, block)) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_backward_slice(T, D, block, a_per_channel, flags, x + s * n,
                                         a + s * na, b + s * n, c + s * n, dy + s * n,
                                         dx + s * n, da + s * na, db + s * n, dc + s * n) != 0;
    return err ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Exact (untruncated) recurrence, Sec. 3 eq. (2.1), with an initial state.  */
/* ------------------------------------------------------------------------ */

int swr_oracle_exact_forward_slice(int64_t T, int64_t D, int a_per_channel, int flags,
                                   const double* x, const double* a, const double* b,
                                   const double* c, const double* h0, double* y,
                                   double* h_last) {
    if (T < 0 || D < 1) return -1;
    if (T > 0 && (!x || !a || !b || !c || !y)) return -1;
    double* s = (double*)malloc((size_t)D * sizeof(double));
    if (!s) return -1;
    for (int64_t mu = 0; mu < D; ++mu) s[mu] = h0 ? h0[mu] : 0.0;
    for (int64_t m = 0; m < T; ++m) {
        for (int64_t mu = 0; mu < D; ++mu) {
            const int64_t e = m * D + mu;
            s[mu] = decay(a, a_per_channel, D, m, mu) * s[mu] + b[e] * x[e];
            y[e] = c[e] * s[mu];
            if (flags & SWR_ORACLE_RESIDUAL) y[e] += x[e];
        }
    }
    if (h_last)
        for (int64_t mu = 0; mu < D; ++mu) h_last[mu] = s[mu];
    free(s);
    return 0;
}

int swr_oracle_exact_backward_slice(int64_t T, int64_t D, int a_per_channel, int flags,
                                    const double* x, const double* a, const double* b,
                                    const double* c, const double* h0, const double* dy,
                                    const double* dh_last, double* dx, double* da,
                                    double* db, double* dc, double* dh0) {
    if (T < 0 || D < 1) return -1;
    if (T > 0 && (!x || !a || !b || !c || !dy || !dx || !da || !db || !dc)) return -1;
    /* Forward again, keeping the state entering every step (pre) and leaving it (post). */
    double* pre = (double*)malloc((size_t)(T * D + D) * sizeof(double));
    double* post = (double*)malloc((size_t)(T * D + D) * sizeof(double));
    double* lam = (double*)malloc((size_t)D * sizeof(double));
    if (!pre || !post || !lam) {
        free(pre); free(post); free(lam);
        return -1;
    }
    for (int64_t mu = 0; mu < D; ++mu) lam[mu] = h0 ? h0[mu] : 0.0; /* lam is the state here */
    for (int64_t m = 0; m < T; ++m) {
        for (int64_t mu = 0; mu < D; ++mu) {
            const int64_t e = m * D + mu;
            pre[e] = lam[mu];
            lam[mu] = decay(a, a_per_channel, D, m, mu) * lam[mu] + b[e] * x[e];
            post[e] = lam[mu];
        }
    }
    if (T > 0) memset(da, 0, (size_t)(a_per_channel ? T * D : T) * sizeof(double));
    /* Reverse sweep: lam = d(loss)/d(state after step m). */
    for (int64_t mu = 0; mu < D; ++mu) lam[mu] = dh_last ? dh_last[mu] : 0.0;
    for (int64_t m = T - 1; m >= 0; --m) {
        for (int64_t mu = 0; mu < D; ++mu) {
            const int64_t e = m * D + mu;
            lam[mu] += c[e] * dy[e];          /* y_m = c_m * state_m            */
            dc[e] = dy[e] * post[e];
            const double du = lam[mu];        /* d state_m / d u_m = 1          */
            dx[e] = b[e] * du;
            if (flags & SWR_ORACLE_RESIDUAL) dx[e] += dy[e];
            db[e] = x[e] * du;
            if (a_per_channel)                /* d state_m / d a_m = state_{m-1} */
                da[e] += lam[mu] * pre[e];
            else
                da[m] += lam[mu] * pre[e];
            lam[mu] *= decay(a, a_per_channel, D, m, mu); /* d state_m / d state_{m-1} */
        }
    }
    if (dh0)
        for (int64_t mu = 0; mu < D; ++mu) dh0[mu] = lam[mu];
    free(pre); free(post); free(lam);
    return 0;
}

int swr_oracle_exact_forward(int64_t S, int64_t T, int64_t D, int a_per_channel, int flags,
                             const double* x, const double* a, const double* b,
                             const double* c, const double* h0, double* y, double* h_last) {
    if (S < 0 || T < 0 || D < 1) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_exact_forward_slice(T, D, a_per_channel, flags, x + s * n, a + s * na,
                                              b + s * n, c + s * n, h0 ? h0 + s * D : NULL,
                                              y + s * n, h_last ? h_last + s * D : NULL) != 0;
    return err ? -1 : 0;
}

int swr_oracle_exact_backward(int64_t S, int64_t T, int64_t D, int a_per_channel, int flags,
                              const double* x, const double* a, const double* b,
                              const double* c, const double* h0, const double* dy,
                              const double* dh_last, double* dx, double* da, double* db,
                              double* dc, double* dh0) {
    if (S < 0 || T < 0 || D < 1) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_exact_backward_slice(
                   T, D, a_per_channel, flags, x + s * n, a + s * na, b + s * n, c + s * n,
                   h0 ? h0 + s * D : NULL, dy + s * n, dh_last ? dh_last + s * D : NULL,
                   dx + s * n, da + s * na, db + s * n, dc + s * n, dh0 ? dh0 + s * D : NULL) != 0;
    return err ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Recurrent form of the jagged window (two states per channel).            */
/* ------------------------------------------------------------------------ */

int swr_oracle_step_slice(int64_t K, int64_t D, int64_t block, int64_t t0, int a_per_channel,
                          int flags, const double* x, const double* a, const double* b,
                          const double* c, double* state, double* y) {
    if (K < 0 || D < 1 || block < 1 || t0 < 0 || !state) return -1;
    if (K > 0 && (!x || !a || !b || !c || !y)) return -1;
    double* e = state;
    double* s = state + D;
    for (int64_t k = 0; k < K; ++k) {
        const int64_t t = t0 + k;
        for (int64_t mu = 0; mu < D; ++mu) {
            const int64_t i = k * D + mu;
            if (t % block == 0) { /* a block starts: the window now reaches back to the
                                     start of the block that just ended */
                e[mu] = s[mu];
                s[mu] = 0.0;
            }
            const double am = decay(a, a_per_channel, D, k, mu);
            const double u = b[i] * x[i];
            e[mu] = am * e[mu] + u;
            s[mu] = am * s[mu] + u;
            y[i] = c[i] * e[mu];
            if (flags & SWR_ORACLE_RESIDUAL) y[i] += x[i];
        }
    }
    return 0;
}

int swr_oracle_step(int64_t S, int64_t K, int64_t D, int64_t block, int64_t t0,
                    int a_per_channel, int flags, const double* x, const double* a,
                    const double* b, const double* c, double* state, double* y) {
    if (S < 0 || K < 0 || D < 1) return -1;
    const int64_t n = K * D, na = a_per_channel ? K * D : K;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_step_slice(K, D, block, t0, a_per_channel, flags, x + s * n, a + s * na,
                                     b + s * n, c + s * n, state + s * 2 * D, y + s * n) != 0;
    return err ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Uniform window: the banded operator of Sec. 4.1 (lags 0 .. k-1).          */
/* ------------------------------------------------------------------------ */

int swr_oracle_uniform_forward_slice(int64_t T, int64_t D, int64_t k, int a_per_channel,
                                     int flags, const double* x, const double* a,
                                     const double* b, const double* c, double* y) {
    if (bad_args(T, D, k)) return -1;
    if (T == 0) return 0;
    if (!x || !a || !b || !c || !y) return -1;
    double* s = (double*)malloc((size_t)D * sizeof(double));
    if (!s) return -1;
    for (int64_t i = 0; i < T; ++i) {
        /* Token i's window: the k most recent tokens, i-k+1 .. i (clipped at 0). */
        const int64_t start = i - k + 1 > 0 ? i - k + 1 : 0;
        for (int64_t mu = 0; mu < D; ++mu) s[mu] = 0.0;
        for (int64_t m = start; m <= i; ++m)
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu;
                s[mu] = decay(a, a_per_channel, D, m, mu) * s[mu] + b[e] * x[e];
            }
        for (int64_t mu = 0; mu < D; ++mu) {
            const int64_t e = i * D + mu;
            y[e] = c[e] * s[mu];
            if (flags & SWR_ORACLE_RESIDUAL) y[e] += x[e];
        }
    }
    free(s);
    return 0;
}

int swr_oracle_uniform_backward_slice(int64_t T, int64_t D, int64_t k, int a_per_channel,
                                      int flags, const double* x, const double* a,
                                      const double* b, const double* c, const double* dy,
                                      double* dx, double* da, double* db, double* dc) {
    if (bad_args(T, D, k)) return -1;
    if (T == 0) return 0;
    if (!x || !a || !b || !c || !dy || !dx || !da || !db || !dc) return -1;
    const int64_t win = k < T ? k : T; /* longest window */
    double* du = (double*)calloc((size_t)(T * D), sizeof(double));
    double* pre = (double*)malloc((size_t)(win * D) * sizeof(double));
    double* lam = (double*)malloc((size_t)D * sizeof(double));
    if (!du || !pre || !lam) {
        free(du); free(pre); free(lam);
        return -1;
    }
    memset(da, 0, (size_t)(a_per_channel ? T * D : T) * sizeof(double));
    for (int64_t i = 0; i < T; ++i) {
        const int64_t start = i - k + 1 > 0 ? i - k + 1 : 0;
        /* Re-run token i's window, keeping the state entering every step. */
        for (int64_t mu = 0; mu < D; ++mu) lam[mu] = 0.0; /* lam is the state here */
        for (int64_t m = start; m <= i; ++m)
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu;
                pre[(m - start) * D + mu] = lam[mu];
                lam[mu] = decay(a, a_per_channel, D, m, mu) * lam[mu] + b[e] * x[e];
            }
        for (int64_t mu = 0; mu < D; ++mu) {   /* y_i = c_i * state_i */
            const int64_t e = i * D + mu;
            dc[e] = dy[e] * lam[mu];
            lam[mu] = c[e] * dy[e];            /* now d(loss)/d(state after step i) */
        }
        for (int64_t m = i; m >= start; --m)
            for (int64_t mu = 0; mu < D; ++mu) {
                const int64_t e = m * D + mu;
                du[e] += lam[mu];              /* d state_m / d u_m = 1          */
                const double g = lam[mu] * pre[(m - start) * D + mu];
                if (a_per_channel)             /* d state_m / d a_m = state_{m-1} */
                    da[e] += g;
                else
                    da[m] += g;
                lam[mu] *= decay(a, a_per_channel, D, m, mu);
            }
    }
    for (int64_t e = 0; e < T * D; ++e) {
        dx[e] = b[e] * du[e];
        if (flags & SWR_ORACLE_RESIDUAL) dx[e] += dy[e];
        db[e] = x[e] * du[e];
    }
    free(du); free(pre); free(lam);
    return 0;
}

int swr_oracle_uniform_forward(int64_t S, int64_t T, int64_t D, int64_t k, int a_per_channel,
                               int flags, const double* x, const double* a, const double* b,
                               const double* c, double* y) {
    if (S < 0 || bad_args(T, D, k)) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_uniform_forward_slice(T, D, k, a_per_channel, flags, x + s * n,
                                                a + s * na, b + s * n, c + s * n, y + s * n) != 0;
    return err ? -1 : 0;
}

int swr_oracle_uniform_backward(int64_t S, int64_t T, int64_t D, int64_t k, int a_per_channel,
                                int flags, const double* x, const double* a, const double* b,
                                const double* c, const double* dy, double* dx, double* da,
                                double* db, double* dc) {
    if (S < 0 || bad_args(T, D, k)) return -1;
    const int64_t n = T * D, na = a_per_channel ? T * D : T;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < S; ++s)
        err |= swr_oracle_uniform_backward_slice(T, D, k, a_per_channel, flags, x + s * n,
                                                 a + s * na, b + s * n, c + s * n, dy + s * n,
                                                 dx + s * n, da + s * na, db + s * n,
                                                 dc + s * n) != 0;
    return err ? -1 : 0;
}

int swr_oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void swr_oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
