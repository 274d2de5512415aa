/*
 * swr.h -- C ABI of the MI355X (gfx950) Sliding Window Recurrence library.
 *
 * The operation (Sliding Window Recurrences, Sec. 4.2: the jagged-window
 * truncation T ~ I_b of the hierarchical decomposition, computed by the Block
 * Two-Pass algorithm, Alg. "Block Two-Pass"): for every batch b and head h,
 * with l = block and token i (0-based) in block tau = floor(i / l),
 *
 *     u_i  = b_i (*) x_i                                   (pre-gate, Sec. 5)
 *     h~_i = sum_{j = l*max(tau-1,0)}^{i} ( prod_{m=j+1}^{i} a_m ) u_j
 *     y_i  = c_i (*) h~_i   (+ x_i if SWR_FLAG_RESIDUAL)   (post-gate, Sec. 5)
 *
 * i.e. the diagonal linear recurrence h_i = a_i h_{i-1} + u_i (Sec. 3,
 * eq. (2.1)) whose state is restarted from zero at the start of the previous
 * block: every token sees its own block and the block before it (lags up to
 * l on a block's first token, up to 2l-1 on its last).  The decay a_i is one
 * scalar per token and head, shared by the head's D channels (Sec. 4.2.2 and
 * Sec. 5, "Featurization"), which makes the intra-block solve a matrix
 * product.  A last block shorter than l behaves as if the inputs were
 * zero-padded at the end.  The initial state is zero.
 *
 * swr_backward returns the exact gradients of that (truncated) forward.
 *
 * Block carriers.  For every block t the forward can save the carrier
 * v_t = w_{t,l}, the last state of the block's local solve started from zero
 * (the "effective input" that the Block Two-Pass algorithm hands to block
 * t+1; the paper suggests checkpointing only this carrier).  They are D
 * float32 values per block: a [B][H][ceil(T/block)][D] array, contiguous,
 * 0.4% of the forward's traffic at D = 128, block = 128.  swr_backward reads
 * them instead of re-reading the previous block's x, b and a; given none, it
 * recomputes each one from those rows itself (the call shape of the paper's
 * problem statement, Alg. "Block Two-Pass": inputs and coefficients only),
 * with the same results bit for bit.  swr_carriers computes them alone.
 *
 * Tensor layout.  x, b, c, y, dy, dx, db, dc are [B, T, H, D] with the channel
 * dimension D contiguous (stride 1) and element strides sx_b, sx_t, sx_h for
 * the other three dimensions (shared by all eight tensors).  a is [B, T, H]
 * with strides sa_b, sa_t, sa_h; da uses the same strides as a but is always
 * float32 (with SWR_FLAG_PER_CHANNEL_DECAY, a and da are [B, T, H, D] with the
 * strides of x instead).  Element type of x, a, b, c, y, dy, dx, db, dc is
 * `dtype`; accumulation is always float32.
 *
 * Ownership.  Every pointer is device memory owned by the caller.  The library
 * allocates no memory.  Its only global state is the static device array that
 * swr_exact_forward_noalloc uses as its workspace (and that array's address
 * per device); every other call keeps no state, and calls from several host
 * threads are safe.  Only the exact-recurrence calls and the backward with
 * shared gates need a workspace, which the caller provides.  Outputs are
 * fully overwritten.
 *
 * Asynchrony.  Work is enqueued on `stream` (a hipStream_t passed as void*;
 * NULL = the default stream) and the call returns without waiting.  A fault
 * inside a kernel surfaces at the caller's next synchronisation.
 *
 * Errors.  Arguments are validated before any HIP runtime call; a failed
 * validation returns a negative SWR_ERR_* code and touches nothing.
 * SWR_ERR_HIP means the kernel launch itself failed.
 */
#ifndef SWR_H
#define SWR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SWR_ABI_VERSION 1

typedef enum swr_status {
    SWR_OK = 0,
    SWR_ERR_NULL = -1,        /* a required pointer is NULL                              */
    SWR_ERR_SHAPE = -2,       /* negative B, T or H, D < 1, or overlapping strides        */
    SWR_ERR_DTYPE = -3,       /* dtype is not one of swr_dtype_t                          */
    SWR_ERR_BLOCK = -4,       /* block is not 16, 32, 64 or 128                           */
    SWR_ERR_ALIGN = -5,       /* a pointer or stride breaks the vector alignment          */
    SWR_ERR_ALIAS = -6,       /* an output overlaps an input or another output            */
    SWR_ERR_UNSUPPORTED = -7, /* D not a multiple of 16 up to 256 (not in {16, 32, 64,
                                 128} outside swr_forward / swr_carriers / swr_backward),
                                 unknown flags, bad run_len, or strides/sizes beyond the
                                 kernels' 32-bit offsets                                  */
    SWR_ERR_HIP = -8,         /* the HIP runtime rejected the launch                      */
    SWR_ERR_VERSION = -9,     /* problem->abi_version != SWR_ABI_VERSION                  */
    SWR_ERR_SCRATCH = -10     /* swr_exact_forward_noalloc: the problem needs more than
                                 SWR_NOALLOC_SCRATCH_BYTES of workspace                    */
} swr_status_t;

typedef enum swr_dtype {
    SWR_DTYPE_F32 = 0,        /* IEEE float32                                            */
    SWR_DTYPE_BF16 = 1        /* bfloat16; outputs are rounded to nearest even            */
} swr_dtype_t;

/* y += x in the forward and dx += dy in the backward (Phalanx post-gate with
 * residual, Sec. 5). */
#define SWR_FLAG_RESIDUAL 1u

/* Per-channel decay: a holds one decay per token, head AND channel, i.e. the
 * diagonal transition a_t (*) h_{t-1} of eq. (2.1) with a full diagonal
 * instead of one scalar per head.  a is then [B, T, H, D] in the I/O dtype
 * and da is [B, T, H, D] float32, both with the strides sx_* of x (sa_* are
 * not read), with the alignment of x (da: of its float32 lane slices, i.e.
 * min(16, 4 * min(D, 64) / 16) bytes).  The window truncation, carriers and
 * every other convention are unchanged; the per-channel da is not summed
 * over channels.  The intra-block solve is then a per-channel scan rather
 * than a matrix product (the operator L_t differs from channel to channel). */
#define SWR_FLAG_PER_CHANNEL_DECAY 2u

/* Fused featurisation (Phalanx layer, Sec. 5, "Featurization": the decay and
 * the key-like pre-gate are sigmoids of linear projections).  With
 * SWR_FLAG_SIGMOID_DECAY, `a` holds logits z_a and the decay is sigmoid(z_a);
 * with SWR_FLAG_SIGMOID_PREGATE, `b` holds logits z_b and the pre-gate is
 * sigmoid(z_b).  The sigmoid is evaluated in float32 from the stored logits.
 * swr_backward then returns da = dL/dz_a and db = dL/dz_b (the gradients
 * with respect to the stored logits).  Either flag combines with the others. */
#define SWR_FLAG_SIGMOID_DECAY 4u
#define SWR_FLAG_SIGMOID_PREGATE 8u

typedef struct swr_problem {
    int32_t abi_version;   /* must be SWR_ABI_VERSION                                     */
    int32_t dtype;         /* swr_dtype_t of every tensor except da                       */
    int64_t B, T, H, D;    /* batch, tokens, heads, channels per head; B, T or H may be 0;
                              D a multiple of 16 up to 256 (see "Head width")             */
    int64_t block;         /* l, the block (= window unit) length: 16, 32, 64 or 128       */
    uint32_t flags;        /* SWR_FLAG_* bits                                              */
    int32_t reserved;      /* must be 0                                                    */
    int64_t sx_b, sx_t, sx_h;  /* element strides of the [B,T,H,D] tensors (channel = 1) */
    int64_t sa_b, sa_t, sa_h;  /* element strides of a and da (ignored with
                                  SWR_FLAG_PER_CHANNEL_DECAY: a, da then use sx_*)      */
    int64_t run_len;       /* tokens per workgroup run: 0 = automatic (chosen separately
                              for the forward and the backward), else a positive multiple
                              of max(64, block) used by both; a tuning knob that does not
                              change results beyond float32 rounding order              */
} swr_problem_t;

/* Head width.  The kernels process heads of W = 16, 32, 64 or 128 channels
 * (a lane holds W/16 channels of a token row).  swr_forward, swr_carriers and
 * swr_backward take any D that is a multiple of 16 up to 256 (the paper's
 * heads are d = D_model / h, Sec. 5): a head wider than 128 channels (64 with
 * SWR_FLAG_PER_CHANNEL_DECAY) runs as 2 (or 4) virtual heads of D/2 (D/4)
 * channels, and a (virtual) head narrower than the next of the widths W
 * leaves the lanes past its channels idle.  With one decay per head, the
 * decay gradient of a head split in two is the sum of the halves' shares,
 * added onto a zeroed da by two float32 atomic adds (the same sum in either
 * order).  Every other entry point takes D in {16, 32, 64, 128}.
 *
 * Forward: y = SWR(x, a, b, c).  Alignment: x, b, c, y and every sx_* must be
 * multiples of min(16 bytes, W/16 elements), W the kernel width above (each
 * lane's slice of a row is a naturally aligned vector; W = D for D in {16,
 * 32, 64, 128}); a needs the alignment of one element.
 * carriers: NULL, or swr_carrier_elems(problem) float32 values (16-byte
 * aligned) that receive the block carriers for swr_backward. */
int swr_forward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                const void* c, void* y, float* carriers, void* stream);

/* Block carriers alone (what swr_forward writes to `carriers`), from x, a, b. */
int swr_carriers(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                 float* carriers, void* stream);

/* Backward: given dy = dL/dy, writes dx, da (float32 with a's shape and strides),
 * db and dc.  x, a, b, c are the forward's inputs.  carriers: the block
 * carriers of those same inputs (from swr_forward or swr_carriers; 16-byte
 * aligned), or NULL, in which case the kernel recomputes the carrier of the
 * block before each of its steps from that block's x, b and a (the rows it
 * processes next; no workspace, no allocation; identical results, at the
 * cost of reading those rows once more).  Nothing else from the forward is
 * needed: the kernel recomputes the local solves it uses. */
int swr_backward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                 const void* c, const void* dy, const float* carriers, void* dx, float* da,
                 void* db, void* dc, void* stream);

/* Number of float32 block carriers of a problem, B * H * ceil(T / block) * D,
 * or a negative SWR_ERR_* code for a problem with invalid shape fields. */
int64_t swr_carrier_elems(const swr_problem_t* problem);

/* Static English description of a status code (never NULL). */
const char* swr_error_string(int code);

/* SWR_ABI_VERSION of the built library. */
int swr_abi_version(void);

/* ------------------------------------------------------------------------
 * Exact (untruncated) recurrence
 *
 * The state sequence of eq. (2.1) with no window truncation and an optional
 * initial state h0:  h_{-1} = h0,  h_i = a_i h_{i-1} + b_i (*) x_i,
 * y_i = c_i (*) h_i (+ x_i with SWR_FLAG_RESIDUAL).  It is the result of the
 * hierarchical decomposition L = calL + G Z_b T R (Sec. 3.2, Thm.
 * "Hierarchical Decomposition") evaluated by Alg. "Hierarchical Block Parallel
 * Inference" in its three stages, at the granularity of a workgroup's run of
 * blocks: (I) local solves of every run from zero, keeping each run's end
 * state and decay product; (II) the carrier recurrence s_r = c_r s_{r-1} + v_r
 * over a sequence's runs; (III) every run again from its exact entering
 * state.  This is the recurrence that the jagged window approximates; with
 * h0 and h_last it also chains a long sequence processed in pieces, and a
 * single-token piece is the recurrent decoding step.  Stages I and III both
 * read their inputs, so the three stages move about 1.5x the bytes of
 * swr_forward (the backward about 1.25x).  Unless heads of 16 or 32
 * channels, stored next to each other with one decay per head, run packed
 * four or two to a 64-channel group, the forward instead runs the three
 * stages in one pass over chunks of 128 tokens, each chunk
 * composing the published aggregates of the chunks before it (a look-back
 * between workgroups in a fixed pattern, so that repeated calls give the same
 * bits): it reads every input once.  The backward does the same, from each
 * sequence's end, for heads of up to 64 channels (one decay per head).  A
 * chunk waits only for chunks that are already running, and gives up after
 * 65536 polls (never expected): it then adds one to the workspace's second
 * 32-bit integer and continues from NaN, so that every output depending on
 * it is NaN rather than a plausible value.  The environment variable
 * SWR_CHAIN_SPIN_LIMIT (read at every call, 0 to 65535) lowers that limit,
 * to exercise this path; it cannot raise it.
 *
 * Everything in swr_problem_t keeps its meaning except that `block` only sets
 * the length of the exact block carriers; every flag applies (with
 * SWR_FLAG_PER_CHANNEL_DECAY the layouts and alignment of a and da are those
 * of swr_forward / swr_backward with that flag).  h0, h_last, dh_last and dh0 are
 * float32 [B][H][D], contiguous, 16-byte aligned; NULL h0 / dh_last mean
 * zero, NULL h_last / dh0 skip that output.
 *
 * Workspace: swr_exact_workspace_bytes(problem) bytes of device memory
 * (16-byte aligned, owned by the caller, needing no initialisation; it may be
 * NULL when that size is 0).  Its contents are scratch and are overwritten;
 * two calls in flight at once need two workspaces.  After a one-pass call's
 * work has completed, its second 32-bit integer holds the number of waits
 * that gave up (see above; 0 in every correct run).
 * ------------------------------------------------------------------------ */

/* Bytes of workspace swr_exact_forward / swr_exact_backward need for this
 * problem, or a negative SWR_ERR_* code. */
int64_t swr_exact_workspace_bytes(const swr_problem_t* problem);

/* Exact forward.  y is required (unless the problem is empty).  carriers:
 * NULL, or swr_carrier_elems(problem) float32 values that receive the exact
 * state at the end of every block ([B][H][ceil(T/block)][D]; a partial last
 * block's entry is the state at token T-1), which swr_exact_backward needs.
 * h_last receives the state after token T-1 (h0 when T = 0). */
int swr_exact_forward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                      const void* c, const float* h0, void* y, float* carriers, float* h_last,
                      void* workspace, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the exact
 * forward with the arguments and results of swr_exact_forward, but with its
 * workspace in a device array that the library owns instead of a caller's
 * buffer.  The call allocates nothing (no hipMalloc, no allocating library
 * routine).  The array is a static device array of SWR_NOALLOC_SCRATCH_BYTES
 * bytes, one per GPU, held from the library's first use of that GPU until the
 * process ends; its address is looked up once per device, on the first call
 * on it.  Where the one-pass forward's workspace exceeds that size and the
 * three stages' does not, the call runs the three stages (the same result up
 * to rounding); a problem for which both exceed it is rejected with
 * SWR_ERR_SCRATCH before any HIP runtime call.  The one-pass
 * forward's publication flags and ticket counters at the start of the array
 * are zeroed by a fill kernel on `stream` at the start of every call (no
 * memset); every other entry is written before it is read.
 * All calls on one GPU share its array: calls whose work overlaps in time on
 * one GPU (different streams, or host threads racing on the same stream)
 * race on it and give wrong results; calls ordered on one stream are safe.
 * Launches go to the device of `stream` (NULL: the current device). */
#define SWR_NOALLOC_SCRATCH_BYTES ((int64_t)32 << 20)
int swr_exact_forward_noalloc(const swr_problem_t* problem, const void* x, const void* a,
                              const void* b, const void* c, const float* h0, void* y,
                              float* carriers, float* h_last, void* stream);

/* Exact backward: gradients of  sum(dy * y) + sum(dh_last * h_last)  with
 * respect to x, a (float32 with a's shape and strides), b, c and h0.  x, a, b,
 * c and h0 are the forward's inputs and `carriers` its exact block carriers
 * (required).  With the sigmoid flags, da and db are with respect to the
 * logits, as in swr_backward. */
int swr_exact_backward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                       const void* c, const void* dy, const float* h0, const float* carriers,
                       const float* dh_last, void* dx, float* da, void* db, void* dc, float* dh0,
                       void* workspace, void* stream);

/* ------------------------------------------------------------------------
 * Recurrent decoding
 *
 * The recurrence processed token by token with a carried state, for
 * generating one (or a few) tokens at a time after a prompt, i.e. decoding
 * the layer as a recurrence (Sec. 6, comparison of Phalanx variants).  problem->T is the
 * number of tokens K in the call (usually 1); x, a, b, c, y hold those K
 * tokens with the usual layouts and strides; every flag applies.  The
 * alignment rules are those of swr_forward without the per-channel flag
 * (a per-channel a then needs the alignment of x).  The state is float32,
 * contiguous, 16-byte aligned, and is read and overwritten in place; K = 0
 * leaves it unchanged.  A thread carries each (batch, head, 16th of the
 * channels) through the K tokens in order: meant for short calls; long
 * prompts go through swr_forward and swr_decode_state.
 * ------------------------------------------------------------------------ */

/* Jagged window.  state is [B][H][2][D]: per channel e, the state restarted
 * at the start of the previous block (what the outputs read), then s, the
 * state restarted at the start of the current block -- both after token t0-1
 * (zeros before the first token).  When a token t with t mod block == 0
 * starts a block, e takes s and s restarts from zero; then e and s both take
 * the step h <- a_t h + b_t x_t and y_t = c_t e (+ x_t).  The outputs are
 * exactly those of swr_forward over the whole sequence (Sec. 4.2's window). */
int swr_step(const swr_problem_t* problem, int64_t t0, const void* x, const void* a, const void* b,
             const void* c, void* y, float* state, void* stream);

/* Exact recurrence: state is h, [B][H][D] (h0 / h_last of swr_exact_forward);
 * h <- a_t h + b_t x_t, y_t = c_t h (+ x_t).  problem->block must be valid but
 * is not used. */
int swr_exact_step(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                   const void* c, void* y, float* state, void* stream);

/* The jagged window's decoding state (swr_step's [B][H][2][D]) after a
 * forward pass over tokens 0 .. T-1 of `problem`, from that pass's block
 * carriers (swr_forward / swr_carriers) and a: s is the carrier of the last
 * (possibly partial) block and e = s + (product of the last block's decays)
 * times the carrier of the block before it. */
int swr_decode_state(const swr_problem_t* problem, const void* a, const float* carriers, float* state,
                     void* stream);

/* ------------------------------------------------------------------------
 * Gates shared by groups of heads
 *
 * The Phalanx layer may share the key-like pre-gate and the query-like
 * post-gate across groups of heads, as grouped-query attention shares keys
 * and values (Sec. 5, "Gate sharing across heads"): heads g*group ..
 * g*group + group - 1 all use b[:, :, g] and c[:, :, g].  b and c (and db,
 * dc) are then [B, T, H / group, D] with element strides gate_strides[0..2]
 * (batch, token, group; the channel stride is 1), alignment as for x.  The
 * recurrence is the jagged window of swr_forward / swr_backward, with the
 * same carriers; db and dc are the gradients with respect to the shared
 * gates (sums over each group's heads, added in head order, so results are
 * reproducible).  For groups of up to 16 heads the backward sums a group's
 * shares inside one pass and needs no workspace; larger groups write every
 * head's float32 shares to a caller-provided workspace, summed in a second
 * launch.  One decay per head only (SWR_FLAG_PER_CHANNEL_DECAY is rejected);
 * heads of 16 and 32 channels are not packed.  group = 1 is the ordinary
 * layout with b, c at their own strides.
 * ------------------------------------------------------------------------ */

/* Workspace bytes swr_backward_shared_gates needs: 0 for groups of up to 16
 * heads, else 2 * B * T * H * D float32 (the heads' shares of db and dc); or a
 * negative SWR_ERR_* code. */
int64_t swr_shared_gates_workspace_bytes(const swr_problem_t* problem, int64_t group);

/* Forward with shared gates: y = SWR(x, a, b, c) where head h reads
 * b[:, :, h / group] and c[:, :, h / group].  carriers as for swr_forward. */
int swr_forward_shared_gates(const swr_problem_t* problem, int64_t group, const int64_t* gate_strides,
                             const void* x, const void* a, const void* b, const void* c, void* y,
                             float* carriers, void* stream);

/* Backward with shared gates: dx, da as for swr_backward; db and dc in the
 * gates' layout.  workspace: swr_shared_gates_workspace_bytes bytes of device
 * memory (16-byte aligned, no initialisation needed, overwritten); may be NULL
 * when that size is 0. */
int swr_backward_shared_gates(const swr_problem_t* problem, int64_t group, const int64_t* gate_strides,
                              const void* x, const void* a, const void* b, const void* c, const void* dy,
                              const float* carriers, void* dx, float* da, void* db, void* dc,
                              void* workspace, void* stream);

/* ------------------------------------------------------------------------
 * Uniform window
 *
 * The other truncation of Sec. 4 (Sec. 4.1, "Uniform Window Recurrences"):
 * the Kogge-Stone factorisation of Sec. 3.1, eq. (2.4), stopped after log2 k
 * stages, i.e. the banded operator  L~ = I + AZ + (AZ)^2 + ... + (AZ)^{k-1}.
 * Every token sees exactly its k most recent tokens:
 *
 *     h~_i = sum_{j = max(0, i-k+1)}^{i} ( prod_{m=j+1}^{i} a_m ) b_j (*) x_j
 *     y_i  = c_i (*) h~_i   (+ x_i if SWR_FLAG_RESIDUAL)
 *
 * The window length k is problem->block (16, 32, 64 or 128; the stage counts
 * 4 .. 7 of the scan).  With the jagged window of the same block, a token
 * sees at least these lags (all of them on a block's first token) and at most
 * those of the uniform window of 2k.  The kernels evaluate it block by block
 * (a local solve plus, for every row, the tail of the previous block that its
 * window still holds), not as the paper's truncated flat scan; nothing is
 * saved between the forward and the backward, which recomputes what it needs
 * from the previous block's x, b and a.  Everything in swr_problem_t keeps its
 * meaning; SWR_FLAG_PER_CHANNEL_DECAY is not supported (SWR_ERR_UNSUPPORTED).
 * Alignment: x, b, c, y, dy, dx, db, dc and every sx_* in multiples of
 * min(16 bytes, min(D, 64)/16 elements); a of one element; da of 4 bytes.
 * ------------------------------------------------------------------------ */

/* Forward: y = the uniform-window recurrence of x, a, b, c. */
int swr_uniform_forward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                        const void* c, void* y, void* stream);

/* Backward: given dy, the exact gradients dx, da (float32, a's shape and
 * strides), db and dc of swr_uniform_forward (with the sigmoid flags, da and
 * db with respect to the logits). */
int swr_uniform_backward(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                         const void* c, const void* dy, void* dx, float* da, void* db, void* dc,
                         void* stream);

/* Launch shape the uniform-window calls pick (run length and workgroups of
 * the forward and of the backward); as swr_launch_info. */
int swr_uniform_launch_info(const swr_problem_t* problem, int64_t* fwd_run_len, int64_t* fwd_workgroups,
                            int64_t* bwd_run_len, int64_t* bwd_workgroups);

/* Resolved launch shape for a problem (for reports and tests): the run length
 * in tokens and the number of workgroups of the forward and of the backward
 * launch (any output pointer may be NULL).  Returns an SWR_ERR_* code for a
 * problem that swr_forward would reject on shape grounds; pointers are not
 * inspected. */
int swr_launch_info(const swr_problem_t* problem, int64_t* fwd_run_len, int64_t* fwd_workgroups,
                    int64_t* bwd_run_len, int64_t* bwd_workgroups);

#ifdef __cplusplus
}
#endif
#endif /* SWR_H */
