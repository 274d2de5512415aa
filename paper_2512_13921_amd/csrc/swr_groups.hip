// swr_groups.hip -- gfx950 backward of the jagged window with the pre-gate b
// and the post-gate c shared by groups of heads (the Phalanx layer's gate
// sharing, Sec. 5).
//
// db and dc of a group are sums over its heads.  A workgroup owns one group
// (and one 64-channel half of it when the heads are wider) for a run of
// tokens and, at every step, goes through the group's heads one after
// another: each head's step is the ordinary jagged-window backward step
// (local solves on the matrix cores, the forward carriers from the saved
// block carriers, the reverse carriers from the step before), and its shares
// of db and dc are added to registers, in head order, before one store per
// group.  So b and c are read and db, dc written once per group, and the
// result does not depend on scheduling.  A head's reverse carriers wait in
// LDS between its steps.  Heads of 128 channels run as two halves (the
// registers of one 8-wave group per compute unit do not hold a whole head's
// accumulators); their decay gradients then meet in da as two float32
// atomic adds onto zero, which give the same sum in either order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swr_device.h"
#include "swr_launch.h"

namespace swr {
namespace {

constexpr int kMaxGroup = 16;   // heads per group whose reverse carriers fit the LDS plan

// Work item: (batch, group, channel half, run).  p.Hv = groups << hshift.
struct GWork {
    int64_t b, g, t_begin, t_end;
    int part;
};

__device__ inline GWork group_work(const Params& p) {
    const uint32_t wid = xcd_remap(blockIdx.x, (uint32_t)p.nwork);
    const uint32_t U = (uint32_t)p.Hv, nruns = (uint32_t)p.nruns;
    const uint32_t v = wid % U, rest = wid / U;
    GWork w;
    w.g = v >> p.hshift;
    w.part = (int)(v & ((1u << p.hshift) - 1));
    w.b = rest / nruns;
    w.t_begin = (int64_t)(rest % nruns) * p.run_len;
    w.t_end = min(w.t_begin + p.run_len, p.T);
    return w;
}

template <class IO, int CPL, int TW, bool FEAT>
__global__ __launch_bounds__(TW * 64, 2) void swr_bwd_grouped_kernel(Params p) {
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;
    constexpr int DV = CPL * SB;       // channels this workgroup covers
    constexpr int STEP = TW * SB;      // whole blocks
    constexpr int ES = IO::ES;
    using R_ = Row<IO, CPL>;
    __shared__ float s_wl[2][TW][DV];              // last row of each sub-block's local solve L u
    __shared__ float s_df[2][TW][DV];              // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_c[2][TW];                   // decay product of each sub-block
    __shared__ float s_rev[2][kMaxGroup][2][DV];   // each head's reverse carriers between steps

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const GWork wk = group_work(p);
    const int l = p.block;
    const int S = l / SB;
    const int smask = S - 1;
    const int K = (int)p.group;
    const int64_t D = (int64_t)DV << p.hshift;     // channels of a head
    const int64_t t_la = min(wk.t_end + (int64_t)l, p.T);
    const int base = lane & 48;

    // The group's gates and gate gradients.
    const int64_t go = (wk.b * p.sg_b + wk.g * p.sg_h + (int64_t)wk.part * DV) * ES;
    const char* bb = (const char*)p.b + go;
    const char* cb = (const char*)p.c + go;
    char* dbb = (char*)p.db + go;
    char* dcb = (char*)p.dc + go;
    const int64_t rs = p.sx_t * ES, gs = p.sg_t * ES, as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t goff = (uint32_t)(4 * grp) * (uint32_t)gs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const bool split = p.hshift > 0;

    // Per head j of the group: its rows of x, dy, dx, its decays and its carriers.
    auto head_x = [&](int j) { return (wk.b * p.sx_b + (wk.g * K + j) * p.sx_h + (int64_t)wk.part * DV) * ES; };
    auto head_a = [&](int j) { return wk.b * p.sa_b + (wk.g * K + j) * p.sa_h; };

    int buf = 0, par = 0;
    // Reverse carriers entering the run's end, per head: zero, or from the halo.
#pragma unroll 1
    for (int j = 0; j < K; ++j) {
        float eps[CPL], pr[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { eps[m] = 0.f; pr[m] = 0.f; }
        if (wk.t_end < p.T) {   // the first block after the run (uniform across the workgroup)
            const int64_t r0 = wk.t_end + tw * SB, tr0 = r0 + 4 * grp;
            const char* dyb = (const char*)p.dy + head_x(j);
            const char* ab = (const char*)p.a + head_a(j) * ES;
            const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * gs), rdy = rsrc(dyb + r0 * rs);
            R_ cr[4], dyr[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool ok = tr0 + r < t_la;
                cr[r].template load<kBwdLoad>(rc, in_range(ok, goff + (uint32_t)(r * gs)));
                dyr[r].template load<kBwdLoad>(rdy, in_range(ok, loff + (uint32_t)(r * rs)));
            }
            float a_n = load_scalar<IO, kBwdDecay>(rsrc(ab + r0 * as), in_range(r0 + n < t_la, aoff));
            if (sig_a) a_n = r0 + n < t_la ? sigmoid(a_n) : 0.0f;
            float LT[4];
            build_decay_transposed(a_n, grp, n, LT);
            const typename Contract<IO>::A At = Contract<IO>::prep(LT);
            const float a0 = shfl(a_n, 0);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float dh[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) dh[q] = dyr[q].get(m) * cr[q].get(m);
                const f32x4 Dn = Contract<IO>::run(At, dh);
                if (grp == 0) s_df[buf][tw][n * CPL + m] = a0 * Dn[0];
            }
            const float cq = shfl(row_prefix_prod(a_n), 15);
            if (lane == 0) s_c[buf][tw] = cq;
            lds_barrier();
#pragma unroll 1
            for (int r = TW - 1; r >= 0; --r) {
                if ((r & smask) == smask) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
                }
                const float c_ = s_c[buf][r];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float df = s_df[buf][r][n * CPL + m];
                    eps[m] = c_ * eps[m] + df;
                    pr[m] = c_ * pr[m] + df;
                }
            }
            buf ^= 1;
        }
        if (tw == 0 && grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_rev[par][j][0][n * CPL + m] = eps[m];
                s_rev[par][j][1][n * CPL + m] = pr[m];
            }
        }
    }
    lds_barrier();

    // One head's inputs for one step: its x and dy rows, its decay (as
    // stored) and the carrier of the block before the step.  Each head's are
    // fetched while the head before it computes.
    struct HeadIn {
        R_ x[4], dy[4];
        float a;
        float v[CPL];
    };
    // (Straight-line code whatever the arguments: with live false every
    // access is out of range and reads zero, so that the loads are issued on
    // one path and not waited for where two paths would join.)
    auto fetch = [&](int64_t kk, int jj, bool live, HeadIn& in) {
        const int64_t t0 = wk.t_begin + kk * STEP, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;
        const int64_t xo = head_x(jj);
        const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs),
                                     rdy = rsrc((const char*)p.dy + xo + r0 * rs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(live && tr0 + r < wk.t_end, loff + (uint32_t)(r * rs));
            in.x[r].template load<kBwdLoad>(rx, o);
            in.dy[r].template load<kBwdLoad>(rdy, o);
        }
        in.a = load_scalar<IO, kBwdDecay>(rsrc((const char*)p.a + (head_a(jj) + r0 * p.sa_t) * ES),
                                          in_range(live && r0 + n < wk.t_end, aoff));
        Row<IoF32, CPL> vr;
        const float* vb = p.carriers + ((wk.b * p.H + wk.g * K + jj) * p.nblocks) * D + (int64_t)wk.part * DV;
        const int64_t blk = (t0 >> p.lshift) - 1;
        vr.load(rsrc(vb), in_range(live && t0 > 0, (uint32_t)(blk * D + n * CPL) * 4u));
#pragma unroll
        for (int m = 0; m < CPL; ++m) in.v[m] = vr.get(m);
    };

    // The gates are fetched a step ahead (PG), each head's inputs a head
    // ahead (PH), where the registers allow it: the featurised and the
    // float32 64-channel kernels would spill.
    constexpr bool PG = CPL <= 2 || (IO::ES == 2 && !FEAT);
    constexpr bool PH = CPL <= 2 || IO::ES == 2 || !FEAT;
    R_ gb[4], gc[4];   // PG: the group's gates of the coming step
    auto fetch_gates = [&](int64_t kk, bool live, R_ (&ob)[4], R_ (&oc)[4]) {
        const int64_t r0 = wk.t_begin + kk * STEP + tw * SB, tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rb = rsrc(bb + r0 * gs), rc = rsrc(cb + r0 * gs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t og = in_range(live && tr0 + r < wk.t_end, goff + (uint32_t)(r * gs));
            ob[r].template load<kBwdLoad>(rb, og);
            oc[r].template load<kBwdLoad>(rc, og);
        }
    };

    const int64_t nsteps = (wk.t_end - wk.t_begin + STEP - 1) / STEP;
    if constexpr (PG) fetch_gates(max(nsteps - 1, (int64_t)0), nsteps > 0, gb, gc);
    HeadIn cur;
    if constexpr (PH) fetch(max(nsteps - 1, (int64_t)0), 0, nsteps > 0, cur);
    for (int64_t k = nsteps - 1; k >= 0; --k, par ^= 1) {
        const int64_t t0 = wk.t_begin + k * STEP;      // a block boundary
        const int64_t r0 = t0 + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
        // The group's gates for this step (with PG fetched during the step
        // before, which then fetches the next step's); the sums of the heads' shares.
        R_ br[4], cr[4];
        if constexpr (PG) {
#pragma unroll
            for (int r = 0; r < 4; ++r) { br[r] = gb[r]; cr[r] = gc[r]; }
            fetch_gates(max(k - 1, (int64_t)0), k > 0, gb, gc);
        } else {
            fetch_gates(k, true, br, cr);
        }
        float sdb[4][CPL], sdc[4][CPL];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) { sdb[r][m] = 0.f; sdc[r][m] = 0.f; }

#pragma unroll 1
        for (int j = 0; j < K; ++j, buf ^= 1) {
            const int64_t xo = head_x(j);
            char* dxb = (char*)p.dx + xo;
            float* const dab = p.da + head_a(j);
            // This head's inputs, fetched while the head before computed; then
            // the next head's (or the next step's first head's).
            if constexpr (!PH) fetch(k, j, true, cur);
            const HeadIn in = cur;
            if constexpr (PH) {
                const bool same = j + 1 < K;   // the next head of this step, else the next step's first
                fetch(same ? k : max(k - 1, (int64_t)0), same ? j + 1 : 0, same || k > 0, cur);
            }
            const R_* const xr = in.x;
            const R_* const dyr = in.dy;
            float a_n = in.a;
            float ds_n = 1.0f;
            if (sig_a) {
                const SigSlope g = sigmoid_slope(a_n);
                ds_n = g.ds;
                a_n = r0 + n < wk.t_end ? g.s : 0.0f;
            }
            const float* const vprev = in.v;   // carrier of the block before this step (zero at the start)

            // ---- local solves W = L u and Dl = L^T dh --------------------------------
            const Decay dk = build_decay(a_n, grp, n);
            f32x4 W[CPL], Dl[CPL];
            {
                const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
                float LT[4];
                build_decay_transposed(a_n, grp, n, LT);
                const typename Contract<IO>::A At = Contract<IO>::prep(LT);
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    float u[4], d4[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
                        d4[q] = dyr[q].get(m) * cr[q].get(m);
                    }
                    W[m] = Contract<IO>::run(A, u);
                    Dl[m] = Contract<IO>::run(At, d4);
                }
            }
            const float a0 = shfl(a_n, 0);
            if (grp == 3) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_wl[buf][tw][n * CPL + m] = W[m][3];
            }
            if (grp == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_df[buf][tw][n * CPL + m] = a0 * Dl[m][0];
            }
            if (lane == 63) s_c[buf][tw] = dk.c;
            lds_barrier();

            // ---- forward carriers entering this wave's sub-block -------------------------
            float ein[CPL], sin_[CPL];
            {
                float e[CPL], s[CPL];
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = vprev[m]; }
#pragma unroll 1
                for (int r = 0; r < tw; ++r) {
                    if ((r & smask) == 0) {
#pragma unroll
                        for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                    }
                    const float c_ = s_c[buf][r];
#pragma unroll
                    for (int m = 0; m < CPL; ++m) {
                        const float wl = s_wl[buf][r][n * CPL + m];
                        e[m] = c_ * e[m] + wl;
                        s[m] = c_ * s[m] + wl;
                    }
                }
                if ((tw & smask) == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                }
#pragma unroll
                for (int m = 0; m < CPL; ++m) { ein[m] = e[m]; sin_[m] = s[m]; }
            }

            // ---- reverse carriers: this head's, from the step after ---------------------
            float eps[CPL], pr[CPL], epsin[CPL], kd = 0.f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                eps[m] = s_rev[par][j][0][n * CPL + m];
                pr[m] = s_rev[par][j][1][n * CPL + m];
            }
#pragma unroll 1
            for (int r = TW - 1; r >= 0; --r) {
                if ((r & smask) == smask) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
                }
                if (r == tw) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) {
                        epsin[m] = eps[m];
                        kd += (ein[m] - sin_[m]) * (eps[m] - pr[m]);
                    }
                }
                const float c_ = s_c[buf][r];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float df = s_df[buf][r][n * CPL + m];
                    eps[m] = c_ * eps[m] + df;
                    pr[m] = c_ * pr[m] + df;
                }
            }
            if (tw == 0 && grp == 0) {   // for this head's next step (the other parity slot)
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    s_rev[par ^ 1][j][0][n * CPL + m] = eps[m];
                    s_rev[par ^ 1][j][1][n * CPL + m] = pr[m];
                }
            }

            // ---- gradients ---------------------------------------------------------------
#pragma unroll
            for (int m = 0; m < CPL; ++m)
#pragma unroll
                for (int r = 0; r < 4; ++r) W[m][r] += dk.G[r] * ein[m];   // the window state H
            float hup[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float v = shfl(W[m][3], (lane - 16) & 63);
                hup[m] = grp == 0 ? ein[m] : v;
            }
            float Rr[4], Gsh[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) Rr[r] = shfl(dk.L[r], base + 15);
            {
                const float gprev = shfl(dk.G[3], (lane - 16) & 63);
                Gsh[0] = grp == 0 ? 1.0f : gprev;
                Gsh[1] = dk.G[0]; Gsh[2] = dk.G[1]; Gsh[3] = dk.G[2];
            }
            const __amdgpu_buffer_rsrc_t rdx = rsrc(dxb + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = tr0 + r;
                float vdx[CPL];
                float acc = -Gsh[r] * Rr[r] * kd;
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float dyv = dyr[r].get(m);
                    sdc[r][m] += dyv * W[m][r];
                    const float du = Dl[m][r] + Rr[r] * epsin[m];
                    const float zb = FEAT ? fresh(br[r].get(m)) : br[r].get(m);
                    const SigSlope g = sig_b ? sigmoid_slope(zb) : SigSlope{zb, 1.0f};
                    vdx[m] = g.s * du;
                    if (p.residual) vdx[m] += dyv;
                    sdb[r][m] += xr[r].get(m) * du * g.ds;
                    acc += (r == 0 ? hup[m] : W[m][r - 1]) * du;
                }
                store_row<IO, CPL, kBwdStore>(rdx, in_range(t < wk.t_end, loff + (uint32_t)(r * rs)), vdx);
                const float tot = row_sum(acc) * shfl(ds_n, base + 4 * grp + r);
                if (n == 0 && t < wk.t_end) {
                    float* dst = dab + t * p.sa_t;
                    if (split)
                        atomicAdd(dst, tot);   // the two halves' shares onto zero
                    else
                        *dst = tot;
                }
            }
        }

        // ---- the group's db and dc for this step ----------------------------------------
        const __amdgpu_buffer_rsrc_t rdb = rsrc(dbb + r0 * gs), rdc = rsrc(dcb + r0 * gs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t og = in_range(tr0 + r < wk.t_end, goff + (uint32_t)(r * gs));
            store_row<IO, CPL, kBwdStore>(rdb, og, sdb[r]);
            store_row<IO, CPL, kBwdStore>(rdc, og, sdc[r]);
        }
    }
}

// Zeroes da ([B, T, H] float32 with a's strides) before two halves add to it.
__global__ __launch_bounds__(256) void swr_grouped_zero_kernel(float* da, int64_t T, int64_t H, int64_t sa_b,
                                                               int64_t sa_t, int64_t sa_h, int64_t total) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int64_t h = i % H, t = (i / H) % T, b = i / (H * T);
    da[b * sa_b + t * sa_t + h * sa_h] = 0.0f;
}

template <class IO, int CPL, bool FEAT>
hipError_t launch_grouped_cpl(const Params& p, int tw, hipStream_t st) {
    const dim3 grid((uint32_t)p.nwork);
    if (tw == 8)
        hipLaunchKernelGGL((swr_bwd_grouped_kernel<IO, CPL, 8, FEAT>), grid, dim3(8 * 64), 0, st, p);
    else if (tw == 4)
        hipLaunchKernelGGL((swr_bwd_grouped_kernel<IO, CPL, 4, FEAT>), grid, dim3(4 * 64), 0, st, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <class IO, bool FEAT>
hipError_t launch_grouped_feat(const Params& p, int cpl, int tw, hipStream_t st) {
    switch (cpl) {
        case 1: return launch_grouped_cpl<IO, 1, FEAT>(p, tw, st);
        case 2: return launch_grouped_cpl<IO, 2, FEAT>(p, tw, st);
        case 4: return launch_grouped_cpl<IO, 4, FEAT>(p, tw, st);
        default: return hipErrorInvalidValue;
    }
}

template <class IO>
hipError_t launch_grouped_io(const Params& p, int cpl, int tw, hipStream_t st) {
    if (p.sig_a || p.sig_b) return launch_grouped_feat<IO, true>(p, cpl, tw, st);
    return launch_grouped_feat<IO, false>(p, cpl, tw, st);
}

}  // namespace

int grouped_max_heads() { return kMaxGroup; }

hipError_t launch_grouped_backward(const Params& p, int dtype, int cpl, int tw, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    if (p.nwork <= 0) return hipSuccess;
    if (p.group < 1 || p.group > kMaxGroup) return hipErrorInvalidValue;
    if (p.hshift > 0) {
        const int64_t total = p.B * p.T * p.H;
        hipLaunchKernelGGL(swr_grouped_zero_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st,
                           p.da, p.T, p.H, p.sa_b, p.sa_t, p.sa_h, total);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return dtype == 1 ? launch_grouped_io<IoBf16>(p, cpl, tw, st) : launch_grouped_io<IoF32>(p, cpl, tw, st);
}

}  // namespace swr
