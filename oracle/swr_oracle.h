/*
 * swr_oracle.h -- reference (oracle) implementation of the Sliding Window
 * Recurrence, forward and backward, in plain C and double precision.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, obviously correct
 * checker that the GPU path is compared against.  Only the test-suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  It shares
 * no code, header, table or helper with the HIP library.
 *
 * What it computes (Sliding Window Recurrences, Sec. 4.2, eqs. for the
 * truncated operator  L~ = calL + G Z_b R  and its block-bidiagonal form):
 * for one (batch, head) slice with T tokens, D channels and block size l,
 * token i (0-based) sits in block tau(i) = floor(i / l) and its window starts at
 * s(i) = l * max(tau(i) - 1, 0).  The state is the scalar recurrence of
 * Sec. 3, eq. (2.1),  h_m = a_m h_{m-1} + u_m,  restarted from zero state at s(i):
 *
 *     h~_i = sum_{j = s(i)}^{i} ( prod_{m = j+1}^{i} a_m ) * u_j ,   u = b (*) x
 *     y_i  = c_i (*) h~_i      (+ x_i when the residual flag is set, Sec. 5
 *                               "post-gate with residual")
 *
 * The forward is literally that restarted loop, one block at a time.  The
 * backward is the exact reverse-mode adjoint of the same loop (the paper gives
 * no backward pass; this is the gradient of the truncated forward).
 *
 * Layouts (per slice, row-major doubles): x, b, c, y, dy, dx, db, dc are
 * [T][D].  a and da are [T] when the decay is shared by the head's D channels
 * (the paper's Phalanx parametrisation, Sec. 5), or [T][D] when per-channel.
 * A last block shorter than l is allowed (equivalent to zero-padding the
 * inputs at the end, Sec. 3.2 assumes n = b*l "for simplicity").
 */
#ifndef SWR_ORACLE_H
#define SWR_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SWR_ORACLE_RESIDUAL 1

/* One slice.  Returns 0, or -1 on a bad argument (T < 0, D < 1, block < 1, NULL). */
int swr_oracle_forward_slice(int64_t T, int64_t D, int64_t block, int a_per_channel,
                             int flags, const double* x, const double* a,
                             const double* b, const double* c, double* y);

/* Gradients of the slice's forward w.r.t. x, a, b, c given dy.  Outputs are
 * overwritten.  da has the shape of a. */
int swr_oracle_backward_slice(int64_t T, int64_t D, int64_t block, int a_per_channel,
                              int flags, const double* x, const double* a,
                              const double* b, const double* c, const double* dy,
                              double* dx, double* da, double* db, double* dc);

/* S independent slices stored back to back ([S][T][D], a as [S][T] or
 * [S][T][D]); slices run in parallel over OpenMP threads.  Returns 0 or -1. */
int swr_oracle_forward(int64_t S, int64_t T, int64_t D, int64_t block, int a_per_channel,
                       int flags, const double* x, const double* a, const double* b,
                       const double* c, double* y);
int swr_oracle_backward(int64_t S, int64_t T, int64_t D, int64_t block, int a_per_channel,
                        int flags, const double* x, const double* a, const double* b,
                        const double* c, const double* dy, double* dx, double* da,
                        double* db, double* dc);

/* The exact (untruncated) recurrence of Sec. 3, eq. (2.1), with an optional
 * initial state: the state sequence that the hierarchical decomposition of
 * Sec. 3.2 (Thm. "Hierarchical Decomposition", Alg. "Hierarchical Block
 * Parallel Inference") computes exactly, and that the window truncation of
 * Sec. 4.2 approximates.  For one slice and channel mu:
 *
 *     h_{-1} = h0 (zero when h0 is NULL),   h_m = a_m h_{m-1} + b_m x_m,
 *     y_m    = c_m h_m   (+ x_m with the residual flag),
 *
 * and h_last = h_{T-1} (h0 itself when T = 0) when h_last is not NULL.
 * h0 and h_last are [D].  Returns 0, or -1 on a bad argument. */
int swr_oracle_exact_forward_slice(int64_t T, int64_t D, int a_per_channel, int flags,
                                   const double* x, const double* a, const double* b,
                                   const double* c, const double* h0, double* y,
                                   double* h_last);

/* Gradients of  L = sum(dy * y) + sum(dh_last * h_last)  for the exact forward
 * above (dh_last NULL means zero): dx, da, db, dc as in the truncated
 * backward, and dh0 = dL/dh0 ([D], skipped when NULL).  The exact
 * reverse-mode adjoint of the forward loop. */
int swr_oracle_exact_backward_slice(int64_t T, int64_t D, int a_per_channel, int flags,
                                    const double* x, const double* a, const double* b,
                                    const double* c, const double* h0, const double* dy,
                                    const double* dh_last, double* dx, double* da,
                                    double* db, double* dc, double* dh0);

/* S slices back to back (as swr_oracle_forward); h0, h_last, dh_last, dh0 are
 * [S][D] or NULL.  Slices run in parallel over OpenMP threads. */
int swr_oracle_exact_forward(int64_t S, int64_t T, int64_t D, int a_per_channel, int flags,
                             const double* x, const double* a, const double* b,
                             const double* c, const double* h0, double* y, double* h_last);
int swr_oracle_exact_backward(int64_t S, int64_t T, int64_t D, int a_per_channel, int flags,
                              const double* x, const double* a, const double* b,
                              const double* c, const double* h0, const double* dy,
                              const double* dh_last, double* dx, double* da, double* db,
                              double* dc, double* dh0);

/* Recurrent (token-by-token) form of the jagged window, with its state: the
 * same outputs as the restarted-window loop above, obtained by carrying two
 * states per channel -- e, the jagged-window state (restarted at the start of
 * the previous block), and s, the state restarted at the start of the current
 * block -- and exchanging them at every block boundary (at a token t with
 * t mod block == 0: e <- s, s <- 0), before the update
 *     e <- a_t e + u_t,  s <- a_t s + u_t,  y_t = c_t e (+ x_t).
 * The K tokens of one call sit at positions t0 .. t0+K-1 of their sequence;
 * `state` ([2][D]: e then s, the state after token t0-1; zeros at t0 = 0) is
 * read and overwritten with the state after the last token.  Returns 0 or -1. */
int swr_oracle_step_slice(int64_t K, int64_t D, int64_t block, int64_t t0, int a_per_channel,
                          int flags, const double* x, const double* a, const double* b,
                          const double* c, double* state, double* y);

/* S slices back to back (x: [S][K][D], a: [S][K] or [S][K][D], state: [S][2][D]). */
int swr_oracle_step(int64_t S, int64_t K, int64_t D, int64_t block, int64_t t0,
                    int a_per_channel, int flags, const double* x, const double* a,
                    const double* b, const double* c, double* state, double* y);

/* Uniform window (Sec. 4.1, "Uniform Window Recurrences"): the Kogge-Stone
 * factorisation of Sec. 3.1 (eq. (2.4)) stopped after log2 k stages keeps the banded
 * operator  L~ = I + AZ + (AZ)^2 + ... + (AZ)^{k-1},  i.e. every token sees
 * exactly the k most recent tokens (lags 0 .. k-1):
 *
 *     h~_i = sum_{j = max(0, i-k+1)}^{i} ( prod_{m=j+1}^{i} a_m ) * u_j ,
 *     y_i  = c_i (*) h~_i   (+ x_i with the residual flag).
 *
 * The forward runs the recurrence restarted from zero at i-k+1 once for every
 * token i (O(T k D)); the backward is the exact reverse-mode adjoint of that
 * loop.  Any k >= 1 is accepted (the kernels take powers of two, the stage
 * counts of the scan).  Layouts and return codes as for the jagged window. */
int swr_oracle_uniform_forward_slice(int64_t T, int64_t D, int64_t k, int a_per_channel,
                                     int flags, const double* x, const double* a,
                                     const double* b, const double* c, double* y);
int swr_oracle_uniform_backward_slice(int64_t T, int64_t D, int64_t k, int a_per_channel,
                                      int flags, const double* x, const double* a,
                                      const double* b, const double* c, const double* dy,
                                      double* dx, double* da, double* db, double* dc);
int swr_oracle_uniform_forward(int64_t S, int64_t T, int64_t D, int64_t k, int a_per_channel,
                               int flags, const double* x, const double* a, const double* b,
                               const double* c, double* y);
int swr_oracle_uniform_backward(int64_t S, int64_t T, int64_t D, int64_t k, int a_per_channel,
                                int flags, const double* x, const double* a, const double* b,
                                const double* c, const double* dy, double* dx, double* da,
                                double* db, double* dc);

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int swr_oracle_max_threads(void);

/* Sets the number of OpenMP threads of later parallel regions (no-op without
 * OpenMP); n < 1 is ignored. */
void swr_oracle_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
