// swr_launch.h -- internal interface between the host API (swr_api.cpp) and
// the gfx950 kernels (swr_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace swr {

// Everything a kernel needs, already validated by the host.  Strides are in
// elements; the channel stride is 1.
struct Params {
    const void* x;
    const void* a;
    const void* b;
    const void* c;
    const void* dy;
    void* y;
    void* dx;
    float* da;
    void* db;
    void* dc;
    float* carriers;    // [B][H][nblocks][D] float32 block carriers v_t (forward: optional output;
                        // backward: input, unused by mode kRecompute)
    int64_t B, T, H;
    int64_t Hv;         // heads the work is split over: H, or H << hshift virtual heads
    int64_t sx_b, sx_t, sx_h;
    int64_t sa_b, sa_t, sa_h;
    int32_t block;      // l (16, 32, 64 or 128)
    int32_t lshift;     // log2(l)
    int32_t residual;   // 0 or 1
    int32_t sig_a;      // 1: a holds logits, the decay is sigmoid(a) (da is then d/d logit)
    int32_t sig_b;      // 1: b holds logits, the pre-gate is sigmoid(b) (db is then d/d logit)
    int32_t hshift;     // log2 of the virtual heads per head: a head of more channels than a
                        // kernel covers (per-channel decay: 64, else 128) is split into 2^hshift
                        // virtual heads of dv channels each
    int32_t dh;         // channels of a (real) head: the row length of the carrier array
    int32_t dv;         // channels of a virtual head (at most the kernel's D = 16 * CPL)
    int32_t nlane;      // lanes n of a 16-lane row that hold channels: dv / CPL (16 when the
                        // virtual head fills the kernel; the others load zeros, store nothing)
    int64_t run_len;    // tokens per workgroup run, a multiple of the step and of l
    int64_t nruns;      // runs per (batch, head) sequence
    int64_t nwork;      // B * H * nruns workgroups
    int64_t nblocks;    // ceil(T / block): carriers per (batch, head)
    // Exact (untruncated) recurrence, computed in three stages (local solves
    // with run aggregates, a carrier scan over runs, reconstruction); the
    // arrays live in the caller's workspace.
    float* agg_v;       // [B*H][nruns][D]: each run's end state started from zero (stage I out)
    float* agg_p;       // [B*H][nruns]: each run's decay product (stage I out); per channel,
                        // [B*H][nruns][D], with a per-channel decay
    const float* carry; // [B*H][nruns][D]: the state entering each run (stage III in); for the
                        // backward, the adjoint entering each run from its end
    const float* h0;    // [B][H][D] initial state (backward stage III), or NULL for zero
    int64_t agg_len;    // stage III: tokens per aggregate run of stage I (this launch's run
                        // length divides by it), and their number per sequence
    int64_t agg_nruns;
    // Gates shared by groups of heads (mode kGrouped): b and c are
    // [B, T, H / group, D] with element strides sg_*; the backward writes
    // every head's share of db and dc, in float32, to gws ([2][B][T][H][D],
    // contiguous), which swr_gate_reduce_kernel then sums over each group.
    int64_t group;
    int64_t sg_b, sg_t, sg_h;
    float* gws;
    // Exact forward in one pass (swr_chain.hip), over the B * Hv virtual
    // sequences of dv channels (dh = D): per chunk of a sequence a
    // publication flag, the chunk's aggregate (agg_v [.][nchunks][dv], agg_p
    // [.][nchunks]) or its inclusive end state; a ticket counter hands out
    // the chunks in order (nruns = chunks per sequence).
    int32_t* chain_flags;   // [B*Hv][nchunks]
    int32_t* chain_ctr;     // [2]: next ticket, look-back time-outs
    int32_t spin_limit;     // polls before a look-back wait gives up
    float* chain_incl;      // [B*Hv][nchunks][dv]
    float* h_last;          // [B][H][D] or NULL
    // Exact backward in one pass: the gradient entering the final state, and
    // the one leaving towards h0 (each [B][H][D] or NULL).
    const float* dh_last;
    float* dh0;
};

// What a forward or backward launch computes.
enum Mode {
    kSwr = 0,        // the jagged-window (truncated) recurrence
    kAggregate = 1,  // exact, stage I: run aggregates only (no outputs)
    kExact = 2,      // exact, stage III: outputs from the carry entering each run
    kGrouped = 3,    // the jagged window with b and c shared by groups of heads
    kPaired = 4,     // the jagged window's forward, two heads of D/2 channels per kernel
                     // head (lanes 0-7 of a 16-lane row hold the first, 8-15 the second)
    kRecompute = 5,  // the jagged window's backward without saved block carriers: each step
                     // recomputes the carrier of the block before it from that block's x, b, a
};

// Sums the per-head float32 shares of db and dc that a kGrouped backward left
// in p.gws over each group of p.group heads, in head order, and writes db and
// dc ([B, T, H / group, D], strides sg_*) in the I/O dtype.
hipError_t launch_gate_reduce(const Params& p, int dtype, int D, void* stream);

// Fused backward with shared gates: one workgroup per (batch, group, channel
// half, run) goes through the group's heads at every step and stores db, dc
// once per group.  p.Hv = (H / group) << hshift work units, 16 * cpl
// channels each, tw waves per workgroup (whole blocks per step).  Groups of
// at most grouped_max_heads() heads.
int grouped_max_heads();
hipError_t launch_grouped_backward(const Params& p, int dtype, int cpl, int tw, void* stream);

// Stage II of the exact recurrence: for every (batch, head) and channel, the
// carrier recurrence over a sequence's runs, S_r = P_r S_{r-1} + V_r forward
// (reverse == 0) or S_r = P_r S_{r+1} + V_r backward, from `init` (or 0);
// carry[r] receives the value entering run r and `fin` (if not NULL) the
// value after the last run.
struct ScanParams {
    const float* agg_v;
    const float* agg_p;
    float* carry;
    const float* init;  // [B*H][D] or NULL
    float* fin;         // [B*H][D] or NULL
    int64_t seqs;       // B * H
    int64_t nruns;
    int32_t D;
    int32_t reverse;
    int32_t p_per_channel;   // agg_p holds one product per channel ([B*H][nruns][D])
};

// Recurrent (token-by-token) steps: K tokens at positions t0 .. t0+K-1 of
// every (batch, head) sequence, carrying the state across calls.  The jagged
// window's state is (e, s) per channel, [B*H][2][D]; the exact recurrence's
// is h, [B*H][D]; both are read and overwritten in place.
struct StepParams {
    const void* x;
    const void* a;
    const void* b;
    const void* c;
    void* y;
    float* state;
    int64_t B, K, H;
    int64_t sx_b, sx_t, sx_h;   // element strides of x, b, c, y (and of a for a per-channel decay)
    int64_t sa_b, sa_t, sa_h;   // element strides of a (one decay per head)
    int64_t t0;                 // sequence position of the first token
    int32_t block;              // l (the jagged window's block length)
    int32_t residual, sig_a, sig_b;
};

// The jagged window's recurrent state after a forward pass over tokens
// 0 .. T-1, from that pass's block carriers and the decays of its last block.
struct StateParams {
    const void* a;
    const float* carriers;      // [B][H][nblocks][D]
    float* state;               // [B*H][2][D]
    int64_t B, T, H;
    int64_t sa_b, sa_t, sa_h;   // strides of a (those of x for a per-channel decay)
    int64_t nblocks;
    int32_t lshift;             // log2(l)
    int32_t sig_a;
};

// Workgroup shape: tw waves per head along the tokens (a step is tw * 16
// tokens) times hw heads of one batch entry (hw must divide H).  The
// backward's steps must hold whole blocks.  Two heads per forward workgroup
// make its loads of the [B, T, H, D] tensors longer contiguous stretches
// (measured 10-13% faster); the backward, whose 256-register waves allow
// only eight per compute unit, measured no faster with two heads and keeps
// one.
struct Shape {
    int tw, hw;
};
inline Shape bwd_shape(int64_t block, int64_t /*H*/) {
    return {block >= 128 ? 8 : 4, 1};
}
inline Shape fwd_shape_single() { return {4, 1}; }
inline Shape fwd_shape(int64_t /*block*/, int64_t H) {
    if (H % 2 == 0) return {2, 2};
    return fwd_shape_single();
}

// Heads of more channels than one kernel head covers are processed as 2^hshift
// virtual heads of D >> hshift channels: at most 64 with a per-channel decay
// (nothing couples the channels there), at most 128 with a decay per head
// (whose decay gradient then sums the virtual heads' shares).
inline int pc_hshift(int64_t D) { return D > 128 ? 2 : D > 64 ? 1 : 0; }
inline int head_hshift(int64_t D) { return D > 128 ? 1 : 0; }

// Launches the forward or backward kernel for (dtype, D, shape) on `stream`;
// for the per-channel kernels D is the channel count of a virtual head.
// pack > 1: a per-head decay with heads of 64 / pack channels, run on the
// per-channel kernels with `pack` adjacent heads per 64-channel virtual head.
hipError_t launch(const Params& p, int dtype, int D, const Shape& shape, bool backward, bool per_channel,
                  int pack, int mode, void* stream);

hipError_t launch_scan(const ScanParams& q, void* stream);

// The exact recurrence's forward in one pass over chunks of chain_tokens()
// tokens (one decay per head): p.nruns chunks per sequence, p.nwork
// persistent workgroups; the workspace arrays of p are reset first.
int chain_tokens();
hipError_t launch_chain_forward(const Params& p, int dtype, int cpl, void* stream);
// The same for bf16 heads of 64 channels taken two at a time (H even; the
// pair's chain uses the per-channel workspace layout with 128 channels).
hipError_t launch_chain_forward_pair(const Params& p, void* stream);
// The same with a decay per channel (virtual heads of 16 * cpl channels).
hipError_t launch_chain_forward_pc(const Params& p, int dtype, int cpl, void* stream);
// The exact recurrence's backward in one pass over the same chunks, taken
// from each sequence's end (heads of 16 * cpl channels, no virtual split;
// p.carriers are the forward's exact block carriers).
hipError_t launch_chain_backward(const Params& p, int dtype, int cpl, void* stream);

// Uniform window of block tokens (the window length): forward or backward
// over 2^hshift virtual heads of 16 * cpl channels per head; the workgroups
// hold 8 waves, 128 / block virtual heads each, and p.nwork is B times the
// number of such head groups (the last one padded) times the runs.
hipError_t launch_uniform(const Params& p, int dtype, int cpl, bool backward, void* stream);

hipError_t launch_step(const StepParams& q, int dtype, int D, bool exact, bool per_channel, void* stream);

hipError_t launch_state(const StateParams& q, int dtype, int D, bool per_channel, void* stream);

}  // namespace swr
