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
    int64_t sx_b, sx_t, sx_h;
    int64_t sa_b, sa_t, sa_h;
    int32_t block;      // l (16, 32, 64 or 128)
    int32_t lshift;     // log2(l)
    int32_t residual;   // 0 or 1
    int64_t run_len;    // tokens per workgroup run, a multiple of the step and of l
    int64_t nruns;      // runs per (batch, head) sequence
    int64_t nwork;      // B * H * nruns workgroups
    int64_t nblocks;    // ceil(T / block): carriers per (batch, head)
};

// Waves per workgroup.  The backward's steps (waves * 16 tokens) must hold
// whole blocks; the forward's need not, and it uses small workgroups so that
// several run side by side on a compute unit.
inline int bwd_waves_for_block(int64_t block) { return block >= 128 ? 8 : 4; }
inline int fwd_waves_for_block(int64_t /*block*/) { return 4; }

// Launches the forward or backward kernel for (dtype, D, waves) on `stream`.
hipError_t launch(const Params& p, int dtype, int D, int nw, bool backward, void* stream);

}  // namespace swr
