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
                        // backward: input)
    int64_t B, T, H;
    int64_t Hv;         // heads the work is split over: H, or H << hshift virtual heads
    int64_t sx_b, sx_t, sx_h;
    int64_t sa_b, sa_t, sa_h;
    int32_t block;      // l (16, 32, 64 or 128)
    int32_t lshift;     // log2(l)
    int32_t residual;   // 0 or 1
    int32_t sig_a;      // 1: a holds logits, the decay is sigmoid(a) (da is then d/d logit)
    int32_t sig_b;      // 1: b holds logits, the pre-gate is sigmoid(b) (db is then d/d logit)
    int32_t hshift;     // per-channel decay: log2 of the virtual heads per head (0 or 1)
    int64_t run_len;    // tokens per workgroup run, a multiple of the step and of l
    int64_t nruns;      // runs per (batch, head) sequence
    int64_t nwork;      // B * H * nruns workgroups
    int64_t nblocks;    // ceil(T / block): carriers per (batch, head)
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

// Per-channel decay: a head is processed as 2^hshift independent virtual
// heads of at most 64 channels (nothing couples the channels there).
inline int pc_hshift(int64_t D) { return D > 64 ? 1 : 0; }

// Launches the forward or backward kernel for (dtype, D, shape) on `stream`;
// for the per-channel kernels D is the channel count of a virtual head.
hipError_t launch(const Params& p, int dtype, int D, const Shape& shape, bool backward, bool per_channel,
                  void* stream);

}  // namespace swr
