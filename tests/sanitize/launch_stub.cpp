// launch_stub.cpp -- host-only stand-ins for the library's kernel launchers,
// so that the C ABI's validation and launch planning (swr_api.cpp) can be
// built for the CPU with AddressSanitizer and UndefinedBehaviorSanitizer and
// driven by the ABI tests.  Test infrastructure: no device code, no HIP
// runtime call.  Every launcher checks the plan it is handed against what
// the kernels assume, then reports that there is no device, as the real
// library does on a machine without a GPU.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../include/swr.h"
#include "../../paper_2512_13921_amd/csrc/swr_internal.h"
#include "../../paper_2512_13921_amd/csrc/swr_launch.h"

namespace {

// A plan the kernels could not execute is a bug in the host code: stop loudly.
void require(bool ok, const char* what) {
    if (!ok) {
        fprintf(stderr, "launch_stub: invalid launch plan: %s\n", what);
        abort();
    }
}

void check_params(const swr::Params& p, int D) {
    require(p.B >= 1 && p.T >= 1 && p.H >= 1, "empty problem launched");
    require(D == 16 || D == 32 || D == 64 || D == 128, "kernel channel count");
    require(p.block == 16 || p.block == 32 || p.block == 64 || p.block == 128, "block");
    require((1 << p.lshift) == p.block, "lshift");
    require(p.run_len > 0 && p.run_len % 16 == 0, "run length");
    require(p.nruns == (p.T + p.run_len - 1) / p.run_len, "run count");
    require(p.nwork >= 1 && p.nwork <= 0x7fffffffLL, "workgroup count");
    require(p.nblocks == (p.T + p.block - 1) / p.block, "block count");
    require(p.Hv >= 1, "virtual heads");
}

// The one-pass chains' poll limit: never above its default of 2^16.  A test
// states the value it expects through SWR_STUB_EXPECT_SPIN_LIMIT.
void check_spin_limit(const swr::Params& p) {
    require(p.spin_limit >= 0 && p.spin_limit <= 65536, "look-back poll limit");
    const char* want = getenv("SWR_STUB_EXPECT_SPIN_LIMIT");
    if (want && *want) require(p.spin_limit == atoi(want), "look-back poll limit not the expected one");
}

}  // namespace

namespace swr {

hipError_t launch(const Params& p, int dtype, int D, const Shape& shape, bool, bool, int pack, int,
                  void*) {
    check_params(p, D);
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(shape.tw >= 1 && shape.hw >= 1 && p.Hv % shape.hw == 0, "workgroup shape");
    require(p.run_len % (shape.tw * 16) == 0, "run length not a multiple of the step");
    require(pack == 1 || pack == 2 || pack == 4, "packing");
    return hipErrorNoDevice;
}

hipError_t launch_scan(const ScanParams& q, void*) {
    require(q.seqs >= 1 && q.nruns >= 1 && q.D >= 1, "scan sizes");
    return hipErrorNoDevice;
}

hipError_t launch_uniform(const Params& p, int dtype, int cpl, bool, void*) {
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(cpl >= 1 && cpl <= 8, "channels per lane");
    require(p.nwork >= 1 && p.nwork <= 0x7fffffffLL, "workgroup count");
    return hipErrorNoDevice;
}

hipError_t launch_step(const StepParams& q, int dtype, int D, bool, bool, void*) {
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(q.B >= 1 && q.K >= 1 && q.H >= 1 && D >= 16, "step sizes");
    return hipErrorNoDevice;
}

hipError_t launch_state(const StateParams& q, int, int D, bool, void*) {
    require(q.B >= 1 && q.H >= 1 && D >= 16, "state sizes");
    return hipErrorNoDevice;
}

hipError_t launch_gate_reduce(const Params& p, int, int D, void*) {
    check_params(p, D);
    require(p.group > 1, "group size");
    return hipErrorNoDevice;
}

int chain_tokens() { return 128; }

hipError_t launch_chain_forward(const Params& p, int dtype, int cpl, void*) {
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(cpl == 1 || cpl == 2 || cpl == 4 || cpl == 8, "channels per lane");
    require(p.nruns == (p.T + 127) / 128 && p.nwork >= 1, "chunks");
    require(p.chain_flags && p.chain_ctr && p.chain_incl && p.agg_v && p.agg_p, "workspace arrays");
    check_spin_limit(p);
    return hipErrorNoDevice;
}

hipError_t launch_chain_forward_pair(const Params& p, void*) {
    require(p.H % 2 == 0 && p.nruns == (p.T + 127) / 128 && p.nwork >= 1, "pairs and chunks");
    require(p.chain_flags && p.chain_ctr && p.chain_incl && p.agg_v && p.agg_p, "workspace arrays");
    check_spin_limit(p);
    return hipErrorNoDevice;
}

hipError_t launch_chain_forward_pc(const Params& p, int dtype, int cpl, void*) {
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(cpl == 1 || cpl == 2 || cpl == 4, "channels per lane");
    require(p.hshift == 0 || cpl == 4, "virtual heads");
    require(p.nruns == (p.T + 127) / 128 && p.nwork >= 1, "chunks");
    require(p.chain_flags && p.chain_ctr && p.chain_incl && p.agg_v && p.agg_p, "workspace arrays");
    check_spin_limit(p);
    return hipErrorNoDevice;
}

hipError_t launch_chain_backward(const Params& p, int dtype, int cpl, void*) {
    require(dtype == SWR_DTYPE_F32 || dtype == SWR_DTYPE_BF16, "dtype");
    require(cpl == 1 || cpl == 2 || cpl == 4 || cpl == 8, "channels per lane");
    require(p.nruns == (p.T + 127) / 128 && p.nwork >= 1, "chunks");
    require(p.chain_flags && p.chain_ctr && p.chain_incl && p.agg_v && p.agg_p, "workspace arrays");
    check_spin_limit(p);
    return hipErrorNoDevice;
}

// Same value as the fused shared-gate backward's limit.
int grouped_max_heads() { return 16; }

hipError_t launch_grouped_backward(const Params& p, int, int cpl, int tw, void*) {
    require(cpl >= 1 && cpl <= 8 && (tw == 4 || tw == 8), "grouped workgroup shape");
    require(p.group >= 1 && p.group <= 16, "group size");
    return hipErrorNoDevice;
}

}  // namespace swr

namespace {
// No device: the static scratch array has no address.
void* no_scratch(void*) { return nullptr; }
}  // namespace

extern "C" int swr_exact_forward_noalloc(const swr_problem_t* problem, const void* x, const void* a,
                                         const void* b, const void* c, const float* h0, void* y,
                                         float* carriers, float* h_last, void* stream) {
    return swr::exact_forward_impl(problem, x, a, b, c, h0, y, carriers, h_last, nullptr, no_scratch,
                                   SWR_NOALLOC_SCRATCH_BYTES, stream);
}
