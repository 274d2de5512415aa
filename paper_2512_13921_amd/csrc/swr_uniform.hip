// swr_uniform.hip -- gfx950 kernels of the uniform-window recurrence.
//
// Method (Sec. 4.1, "Uniform Window Recurrences"): stopping the Kogge-Stone
// factorisation of Sec. 3.1 (eq. (2.4)) after log2 k stages leaves the banded
// operator I + AZ + ... + (AZ)^{k-1}, so every token sees exactly its k most
// recent tokens:
//
//     h_i = sum_{j = i-k+1}^{i} a_{i:j+1} u_j ,   u = b (*) x ,   y_i = c_i (*) h_i .
//
// The paper evaluates it with the truncated flat scan: log2 k passes over the
// whole sequence.  Here the sequence is cut into blocks of l = k tokens and
// each token's window is split at its block start: for token i at offset p
// of block t, the window holds offsets 0 .. p of block t and p+1 .. l-1 of
// block t-1, so
//
//     h_i = (L_t u_t)[p] + g_t[p] Q_{t-1}[p],    Q_{t-1}[p] = sum_{j > p} r_{t-1,j} u_{t-1,j},
//
// with L_t the block's lower-triangular decay operator, g_t its prefix
// products and r_{t-1,j} = a_{j+1} ... a_{end of block t-1}.  Unlike the
// jagged window's rank-one carrier g_t v_{t-1}, the correction Q_{t-1} is a
// whole l x d tile: every row keeps a different tail of the previous block.
//
// Mapping.  A workgroup owns HW (virtual) heads of one batch entry and a run
// of blocks; wave (head, s) owns sub-block s (16 tokens) of every block of its
// head, so a step is one block and the same wave sees the same rows of
// consecutive blocks.  Lanes, MFMA tiles and the hierarchical composition of
// sub-blocks through LDS are those of the jagged-window kernels.  Within a
// sub-block s of a block, Q splits as
//
//     Q[16 s + q] = A_s T_s[q] + V_s,    T_s[q] = sum_{q < j < 16} r^(s)_j u_j
//
// (T_s the sub-block's strict suffix solve, an MFMA with the masked operator
// S[q][j] = r^(s)_j [j > q]; A_s the product of the decays of the block's
// later sub-blocks, V_s their last local rows carried to the block's end).
// The forward keeps its rows of Q in registers from one block to the next;
// a run that does not start its sequence first sweeps the block before it.
//
// Backward (not given in the paper; derived from the forward above).  With
// dh = c (*) dy, D_t = L_t^T dh_t, and C'_{t+1}[p] = sum_{q < p} g_{t+1}[q]
// dh_{t+1,q} (an exclusive prefix of the next block's g-weighted adjoint):
//
//     du_t[p] = D_t[p] + R_t[p] C'_{t+1}[p]        (R_t[p] = a_{p+1} ... a_{l-1} of block t)
//     da_m    = sum_mu  w_t[p-1] D_t[p] + G_t[p-1] E_t[p] + R_t[p] F_t[p-1]
//
// for token m at offset p of block t, where w_t = L_t u_t is the block's local
// state, E_t = L_t^T (dh_t (*) Q_{t-1}), F_t = L_t (u_t (*) C'_{t+1}), and
// w_t[-1] = F_t[-1] = 0, G_t[-1] = 1.  The three terms are the pairs (j, i)
// of window entries that contain a_m (j < m <= i, i - j < l): both in block
// t; j in block t-1 and i in block t; j in block t and i in block t+1.  The
// backward sweeps each run from its last block to its first; every step reads
// block t and the x, b, a of block t-1 (to rebuild Q_{t-1}, the block that
// the next step reads again) and carries its rows of C' to the step before.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swr_device.h"
#include "swr_launch.h"

namespace swr {
namespace {

// A uniform-window work item: a (batch, virtual head, run).  Heads of more
// than 64 channels run as 2^hshift independent 64-channel virtual heads; the
// last group of HW virtual heads may hold padding heads (valid == false),
// which load nothing and store nothing.
struct UWork {
    int64_t b, head, t_begin, t_end;
    int part;
    bool valid;
};

template <int HW>
__device__ inline UWork uni_work(const Params& p, int hw) {
    const uint32_t wid = xcd_remap(blockIdx.x, (uint32_t)p.nwork);
    const uint32_t G = (uint32_t)((p.Hv + HW - 1) / HW), nruns = (uint32_t)p.nruns;
    const int64_t v = (int64_t)(wid % G) * HW + hw;
    const uint32_t rest = wid / G;
    UWork w;
    w.valid = v < p.Hv;
    const int64_t vv = w.valid ? v : 0;
    w.head = vv >> p.hshift;
    w.part = (int)(vv & ((1 << p.hshift) - 1));
    w.b = rest / nruns;
    w.t_begin = (int64_t)(rest % nruns) * p.run_len;
    w.t_end = min(w.t_begin + p.run_len, p.T);
    return w;
}

// Operand A of the strict suffix solve T[q] = sum_{k > q} r_k u_k of a
// sub-block (r_k = a_{k+1} ... a_15): this lane holds S[n][4 grp + q] =
// r_{4 grp + q} when 4 grp + q > n, else 0.  rrow[q] receives r_{4 grp + q}.
__device__ inline void build_suffix_operator(float a_n, int grp, int n, float (&S)[4], float (&rrow)[4]) {
    const float r_n = row_suffix_prod(dpp<DPP_ROW_SHL + 1>(a_n, 1.0f));   // a_{n+1} ... a_15
    const int base = (threadIdx.x & 63) & 48;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int k = 4 * grp + q;
        rrow[q] = shfl(r_n, base + k);
        S[q] = k > n ? rrow[q] : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------

template <class IO, int CPL, int TW, int HW>
__global__ __launch_bounds__(TW * HW * 64, 2) void swr_uni_fwd_kernel(Params p) {
    // Featurisation flags, read at run time (compiling them out measured
    // slower for this kernel, unlike the backward).
    const bool sig_a = p.sig_a, sig_b = p.sig_b;
    // Both contractions take fp32 operands (the fp32 MFMA) whatever the I/O
    // type: this kernel is bound by its VALU work, which the bf16 hi/lo
    // operand split adds to, more than by MFMA cycles.
    using Ct = Contract<IoF32>;
    constexpr int NW = TW * HW;
    constexpr int DV = CPL * SB;    // channels of a virtual head
    constexpr int L = TW * SB;      // block length = window length
    constexpr int ES = IO::ES;
    using RW = Row<IO, CPL>;
    __shared__ float s_wl[2][NW][DV];   // last row of each sub-block's local solve
    __shared__ float s_c[2][NW];        // each sub-block's decay product

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, sg = wv % TW;   // head within the group, sub-block within the block
    const UWork wk = uni_work<HW>(p, hw);

    const int64_t xo = (wk.b * p.sx_b + wk.head * p.sx_h + (int64_t)wk.part * DV) * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    char* yb = (char*)p.y + xo;
    const char* ab = (const char*)p.a + (wk.b * p.sa_b + wk.head * p.sa_h) * ES;
    const int64_t rs = p.sx_t * ES, as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;

    // Q_{t-1} at this lane's rows (zero before the first block).
    float Q[4][CPL];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int m = 0; m < CPL; ++m) Q[r][m] = 0.f;

    // A run that does not start its sequence first sweeps the block before it.
    const int64_t t_first = wk.t_begin > 0 ? wk.t_begin - L : 0;
    int buf = 0;
    for (int64_t t0 = t_first; t0 < wk.t_end; t0 += L, buf ^= 1) {
        const bool halo = t0 < wk.t_begin;
        const int64_t r0 = t0 + sg * SB;          // first token of this wave's sub-block
        const int64_t tr0 = r0 + 4 * grp;         // first of this lane's four tokens
        RW xr[4], br[4], cr[4];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs),
                                         rc = rsrc(cb + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool ok = wk.valid && tr0 + r < wk.t_end;
                const uint32_t o = loff + (uint32_t)(r * rs);
                xr[r].template load<kFwdLoad>(rx, in_range(ok, o));
                br[r].template load<kFwdLoad>(rb, in_range(ok, o));
                cr[r].template load<kFwdLoad>(rc, in_range(ok && !halo, o));
            }
        }
        const bool a_ok = wk.valid && r0 + n < wk.t_end;
        float a_n = load_scalar<IO, kFwdDecay>(rsrc(ab + r0 * as), in_range(a_ok, aoff));
        if (sig_a) a_n = a_ok ? sigmoid(a_n) : 0.0f;
        // (rows past the end of the sequence have u = 0 and reach no output)

        // ---- local solve W = L u and strict suffix solve T = S u ------------
        const Decay dk = build_decay(a_n, grp, n);
        float S[4], rrow[4];
        build_suffix_operator(a_n, grp, n, S, rrow);
        f32x4 W[CPL], Ts[CPL];
        {
            const typename Ct::A AL = Ct::prep(dk.L);
            const typename Ct::A AS = Ct::prep(S);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
                W[m] = Ct::run(AL, u);
                Ts[m] = Ct::run(AS, u);
            }
        }
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[buf][wv][n * CPL + m] = W[m][3];
        }
        if (lane == 63) s_c[buf][wv] = dk.c;
        lds_barrier();

        // ---- the block's earlier sub-blocks (state entering this one, their
        //      decay product) and later ones (the tail that Q carries) -------
        float s[CPL], V[CPL], gp = 1.0f, ra = 1.0f;
#pragma unroll
        for (int m = 0; m < CPL; ++m) { s[m] = 0.f; V[m] = 0.f; }
#pragma unroll 1
        for (int r = 0; r < sg; ++r) {
            const int src = hw * TW + r;
            const float c_ = s_c[buf][src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) s[m] = c_ * s[m] + s_wl[buf][src][n * CPL + m];
            gp *= c_;
        }
#pragma unroll 1
        for (int r = TW - 1; r > sg; --r) {
            const int src = hw * TW + r;
#pragma unroll
            for (int m = 0; m < CPL; ++m) V[m] += ra * s_wl[buf][src][n * CPL + m];
            ra *= s_c[buf][src];
        }

        // ---- outputs: h = W + g (s + G_<s Q_{t-1}) --------------------------
        if (!halo) {
            const __amdgpu_buffer_rsrc_t ry = rsrc(yb + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float yv[CPL];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    yv[m] = cr[r].get(m) * (W[m][r] + dk.G[r] * (s[m] + gp * Q[r][m]));
                    if (p.residual) yv[m] += xr[r].get(m);
                }
                store_row<IO, CPL, kFwdStore>(
                    ry, in_range(wk.valid && tr0 + r < wk.t_end, loff + (uint32_t)(r * rs)), yv);
            }
        }
        // ---- this block's tail tile for the next block ------------------------
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) Q[r][m] = ra * Ts[m][r] + V[m];
    }
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------

template <class IO, int CPL, int TW, int HW, bool FEAT>
__global__ __launch_bounds__(TW * HW * 64, 2) void swr_uni_bwd_kernel(Params p) {
    // Featurisation flags; off at compile time unless FEAT.
    const bool sig_a = FEAT && p.sig_a, sig_b = FEAT && p.sig_b;
    constexpr int NW = TW * HW;
    constexpr int DV = CPL * SB;
    constexpr int L = TW * SB;
    constexpr int ES = IO::ES;
    using RW = Row<IO, CPL>;
    // Per sub-block quantities exchanged through LDS (block t unless noted),
    // double buffered by step; one struct, so that one base address serves all.
    struct Exchange {
        float wl[NW][DV];   // last row of the local solve L u
        float df[NW][DV];   // g-weighted column sum of dh
        float wp[NW][DV];   // block t-1: last row of its local solve
        float de[NW][DV];   // g-weighted column sum of dh * Q_{t-1}
        float wf[NW][DV];   // last row of the local solve L (u * C'_{t+1})
        float c[NW];        // decay product
        float cp[NW];       // block t-1: decay product
    };
    __shared__ Exchange s_x[2];
    // x and b rows of the step's block.  Block t-1's rows, which a step reads
    // for the previous block's tail, are the next step's own: each lane keeps
    // them in LDS slots of its own (no barrier involved) instead of reading
    // them again.
    __shared__ uint32_t s_xb[2][4][RW::NWORDS][NW * 64];
    const int tid = threadIdx.x;

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, sg = wv % TW;
    const UWork wk = uni_work<HW>(p, hw);
    const int base = lane & 48;

    const int64_t xo = (wk.b * p.sx_b + wk.head * p.sx_h + (int64_t)wk.part * DV) * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    const char* dyb = (const char*)p.dy + xo;
    char* dxb = (char*)p.dx + xo;
    char* dbb = (char*)p.db + xo;
    char* dcb = (char*)p.dc + xo;
    const int64_t ao = wk.b * p.sa_b + wk.head * p.sa_h;
    const char* ab = (const char*)p.a + ao * ES;
    float* const dab = p.da + ao;
    const int64_t rs = p.sx_t * ES, as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const bool split = p.hshift > 0;   // da sums channels of several virtual heads

    // Loads the decay of token r0 + n (0 outside [lo, hi)); ds receives its
    // derivative with respect to the stored value (1, or sigma' for a logit).
    auto load_decay = [&](int64_t r0, int64_t lo, int64_t hi, float& ds) {
        const bool ok = wk.valid && r0 + n >= lo && r0 + n < hi;
        float v = load_scalar<IO, kBwdDecay>(rsrc(ab + max(r0, (int64_t)0) * as), in_range(ok, aoff));
        ds = 1.0f;
        if (sig_a) {
            const SigSlope g = sigmoid_slope(v);
            ds = g.ds;
            v = g.s;
        }
        return ok ? v : 0.0f;
    };

    // C'_{t+1} at this lane's rows, for the block the next step processes
    // (kept from one step to the next in this lane's own LDS slots).
    __shared__ float s_cn[4][NW * 64][CPL];
    auto set_cn = [&](int r, const float (&v)[CPL]) {
#pragma unroll
        for (int m = 0; m < CPL; ++m) s_cn[r][tid][m] = v[m];
    };
    {
        float z[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) z[m] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) set_cn(r, z);
    }
    int buf = 0;

    // From block t (g prefix products G, sub-block product c) and its dh:
    // the exclusive prefix Pe[q] = sum_{j < q} g_j dh_j, and (into LDS) the
    // column sum sum_j g_j dh_j.  After the barrier, C' of this wave's rows.
    auto c_prime = [&](const Decay& dk, const float (&dh)[4][CPL], f32x4 (&Pe)[CPL]) {
        float P[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) P[q] = 4 * grp + q < n ? dk.G[q] : 0.0f;
        const typename Contract<IO>::A AP = Contract<IO>::prep(P);
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            float d4[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) d4[q] = dh[q][m];
            Pe[m] = Contract<IO>::run(AP, d4);
            if (grp == 3) s_x[buf].df[wv][n * CPL + m] = Pe[m][3] + dk.G[3] * dh[3][m];
        }
    };
    // Prefix over this head's sub-blocks before sg of the column sums: X = sum_{r < sg} G_<r df_r.
    auto prefix_df = [&](float (&X)[CPL], float& gp) {
#pragma unroll
        for (int m = 0; m < CPL; ++m) X[m] = 0.f;
        gp = 1.0f;
#pragma unroll 1
        for (int r = 0; r < sg; ++r) {
            const int src = hw * TW + r;
#pragma unroll
            for (int m = 0; m < CPL; ++m) X[m] += gp * s_x[buf].df[src][n * CPL + m];
            gp *= s_x[buf].c[src];
        }
    };

    // ---- halo: C' of the block after the run --------------------------------
    if (wk.t_end < p.T) {
        const int64_t r0 = wk.t_end + sg * SB, tr0 = r0 + 4 * grp;
        const int64_t t_hi = min(wk.t_end + (int64_t)L, p.T);
        float dh[4][CPL];
        {
            const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = in_range(wk.valid && tr0 + r < t_hi, loff + (uint32_t)(r * rs));
                RW cr, dyr;
                cr.template load<kBwdLoad>(rc, o);
                dyr.template load<kBwdLoad>(rdy, o);
#pragma unroll
                for (int m = 0; m < CPL; ++m) dh[r][m] = dyr.get(m) * cr.get(m);
            }
        }
        float ds_unused;
        const float a_n = load_decay(r0, 0, t_hi, ds_unused);
        const Decay dk = build_decay(a_n, grp, n);
        f32x4 Pe[CPL];
        c_prime(dk, dh, Pe);
        if (lane == 63) s_x[buf].c[wv] = dk.c;
        lds_barrier();
        float X[CPL], gp;
        prefix_df(X, gp);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float v[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) v[m] = X[m] + gp * Pe[m][r];
            set_cn(r, v);
        }
        buf ^= 1;
    }

    const int64_t nsteps = (wk.t_end - wk.t_begin + L - 1) / L;
    if (nsteps > 0) {   // x and b of the run's last block into this lane's slots
        const int64_t r0 = wk.t_begin + (nsteps - 1) * L + sg * SB, tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t oc = in_range(wk.valid && tr0 + r < wk.t_end, loff + (uint32_t)(r * rs));
            RW xv, bv;
            xv.template load<kBwdLoad>(rx, oc);
            bv.template load<kBwdLoad>(rb, oc);
#pragma unroll
            for (int i = 0; i < RW::NWORDS; ++i) {
                s_xb[0][r][i][tid] = xv.w[i];
                s_xb[1][r][i][tid] = bv.w[i];
            }
        }
    }
    for (int64_t k = nsteps - 1; k >= 0; --k, buf ^= 1) {
        const int64_t t0 = wk.t_begin + k * L;    // a block boundary
        const int64_t r0 = t0 + sg * SB, tr0 = r0 + 4 * grp;
        const int64_t rp = r0 - L;                // the same sub-block of block t-1
        // The rows' offsets, recomputed every step (one add each) rather than
        // kept across the loop: an empty asm hides that lo equals loff.
        uint32_t lo = loff;
        asm volatile("" : "+v"(lo));

        // ---- loads: block t, and x, b, a of block t-1 -----------------------------
        RW xr[4], br[4], dyr[4];
        float dh[4][CPL], up[4][CPL];
        {
            RW cr[4];
            const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs);
            const int64_t rpb = max(rp, (int64_t)0);   // (rows before the sequence are masked)
            const __amdgpu_buffer_rsrc_t rxp = rsrc(xb + rpb * rs), rbp = rsrc(bb + rpb * rs);
            RW xp[4], bp[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = lo + (uint32_t)(r * rs);
                const uint32_t oc = in_range(wk.valid && tr0 + r < wk.t_end, o);
                const uint32_t opv = in_range(wk.valid && rp + 4 * grp + r >= 0, o);
#pragma unroll
                for (int i = 0; i < RW::NWORDS; ++i) {
                    xr[r].w[i] = s_xb[0][r][i][tid];
                    br[r].w[i] = s_xb[1][r][i][tid];
                }
                cr[r].template load<kBwdLoad>(rc, oc);
                dyr[r].template load<kBwdLoad>(rdy, oc);
                xp[r].template load<kBwdLoad>(rxp, opv);
                bp[r].template load<kBwdLoad>(rbp, opv);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int i = 0; i < RW::NWORDS; ++i) {
                    s_xb[0][r][i][tid] = xp[r].w[i];
                    s_xb[1][r][i][tid] = bp[r].w[i];
                }
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    dh[r][m] = dyr[r].get(m) * cr[r].get(m);          // dh = dy * c
                    up[r][m] = xp[r].get(m) * pregate(bp[r].get(m), sig_b);
                }
        }
        float ds_n, ds_unused;
        const float a_n = load_decay(r0, 0, wk.t_end, ds_n);
        const float ap_n = load_decay(rp, 0, wk.t_end, ds_unused);

        // ---- block t: W = L u, Dl = L^T dh, Pe; block t-1: T' = S' u' --------------
        const Decay dk = build_decay(a_n, grp, n);
        float rrow[4];   // r_q of this lane's rows: a_{q+1} ... a_15 of the sub-block
        f32x4 W[CPL], Dl[CPL], Pe[CPL], Tp[CPL];
        float wp0[CPL];
        // L and L^T as MFMA operands, kept for the step's second solves
        // (rebuilt for them in the featurised kernel, which has no registers
        // to spare)
        typename Contract<IO>::A AL, ALT;
        auto prep_L = [&] {
            float LT[4];
            build_decay_transposed(a_n, grp, n, LT);
            AL = Contract<IO>::prep(dk.L);
            ALT = Contract<IO>::prep(LT);
        };
        prep_L();
        {
            float S[4];
            build_suffix_operator(a_n, grp, n, S, rrow);
            float Sp[4], rrow_p[4];
            build_suffix_operator(ap_n, grp, n, Sp, rrow_p);
            const typename Contract<IO>::A ASp = Contract<IO>::prep(Sp);
            c_prime(dk, dh, Pe);
            const float rp0 = shfl(rrow_p[0], base);   // r'_0 (lane n = 0 holds row 0's value)
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4], d4[4], u4p[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
                    d4[q] = dh[q][m];
                    u4p[q] = up[q][m];
                }
                W[m] = Contract<IO>::run(AL, u);
                Dl[m] = Contract<IO>::run(ALT, d4);
                Tp[m] = Contract<IO>::run(ASp, u4p);
                wp0[m] = Tp[m][0] + rp0 * up[0][m];   // block t-1: last local row (grp 0 lanes)
            }
        }
        const float cp = shfl(row_prefix_prod(ap_n), base + 15);
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_x[buf].wl[wv][n * CPL + m] = W[m][3];
        }
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_x[buf].wp[wv][n * CPL + m] = wp0[m];
        }
        if (lane == 63) { s_x[buf].c[wv] = dk.c; s_x[buf].cp[wv] = cp; }
        lds_barrier();

        // ---- the block's other sub-blocks -------------------------------------------
        float s[CPL], X[CPL], pin[CPL], Vp[CPL];
        float gp, ra = 1.0f, rap = 1.0f;
        prefix_df(X, gp);
#pragma unroll
        for (int m = 0; m < CPL; ++m) { s[m] = 0.f; pin[m] = 0.f; Vp[m] = 0.f; }
#pragma unroll 1
        for (int r = 0; r < sg; ++r) {   // state entering this sub-block, restarted at the block start
            const int src = hw * TW + r;
            const float c_ = s_x[buf].c[src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) s[m] = c_ * s[m] + s_x[buf].wl[src][n * CPL + m];
        }
#pragma unroll 1
        for (int r = TW - 1; r > sg; --r) {   // adjoint entering from the block's later sub-blocks
            const int src = hw * TW + r;
            const float c_ = s_x[buf].c[src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                pin[m] = c_ * pin[m] + s_x[buf].df[src][n * CPL + m];
                Vp[m] += rap * s_x[buf].wp[src][n * CPL + m];
            }
            ra *= c_;
            rap *= s_x[buf].cp[src];
        }

        // ---- gradients of x, b, c ----------------------------------------------------
        // Q = Q_{t-1} at this lane's rows; H the window state; D = L_t^T dh;
        // du = D + R C'_{t+1}.
        float Rv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Rv[r] = rrow[r] * ra;
        f32x4 El[CPL], Fl[CPL];
        {
            const __amdgpu_buffer_rsrc_t rdx = rsrc(dxb + r0 * rs), rdb = rsrc(dbb + r0 * rs),
                                         rdc = rsrc(dcb + r0 * rs);
            float vdx[4][CPL], vdb[4][CPL], vdc[4][CPL], eh[4][CPL], uc[4][CPL];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float Cn[CPL], Cnext[CPL];
#pragma unroll
                for (int m = 0; m < CPL; ++m) Cn[m] = s_cn[r][tid][m];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float Qv = rap * Tp[m][r] + Vp[m];
                    const float Hv = W[m][r] + dk.G[r] * (s[m] + gp * Qv);
                    const float Dv = Dl[m][r] + rrow[r] * pin[m];
                    const float du = Dv + Rv[r] * Cn[m];
                    const float dyv = dyr[r].get(m);
                    const float zb = br[r].get(m);
                    const SigSlope g = sig_b ? sigmoid_slope(zb) : SigSlope{zb, 1.0f};
                    vdc[r][m] = dyv * Hv;
                    vdx[r][m] = g.s * du + (p.residual ? dyv : 0.0f);
                    vdb[r][m] = xr[r].get(m) * du * g.ds;
                    eh[r][m] = dh[r][m] * Qv;
                    uc[r][m] = xr[r].get(m) * g.s * Cn[m];
                    Dl[m][r] = Dv;                          // keep D for the decay gradient
                    W[m][r] += dk.G[r] * s[m];              // and the block-restarted state w
                    Cnext[m] = X[m] + gp * Pe[m][r];        // C'_t for the next step
                }
                set_cn(r, Cnext);
                const uint32_t o = in_range(wk.valid && tr0 + r < wk.t_end, lo + (uint32_t)(r * rs));
                store_row<IO, CPL, kBwdStore>(rdx, o, vdx[r]);
                store_row<IO, CPL, kBwdStore>(rdb, o, vdb[r]);
                store_row<IO, CPL, kBwdStore>(rdc, o, vdc[r]);
            }
            if constexpr (FEAT) prep_L();
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float e4[4], f4[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) { e4[q] = eh[q][m]; f4[q] = uc[q][m]; }
                El[m] = Contract<IO>::run(ALT, e4);
                Fl[m] = Contract<IO>::run(AL, f4);
            }
        }
        const float a0 = shfl(a_n, base);
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_x[buf].de[wv][n * CPL + m] = a0 * El[m][0];
        }
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_x[buf].wf[wv][n * CPL + m] = Fl[m][3];
        }
        lds_barrier();
        float pinE[CPL], sF[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { pinE[m] = 0.f; sF[m] = 0.f; }
#pragma unroll 1
        for (int r = 0; r < sg; ++r) {
            const int src = hw * TW + r;
            const float c_ = s_x[buf].c[src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) sF[m] = c_ * sF[m] + s_x[buf].wf[src][n * CPL + m];
        }
#pragma unroll 1
        for (int r = TW - 1; r > sg; --r) {
            const int src = hw * TW + r;
            const float c_ = s_x[buf].c[src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) pinE[m] = c_ * pinE[m] + s_x[buf].de[src][n * CPL + m];
        }

        // ---- decay gradient --------------------------------------------------------
        // da_m = sum_mu w[p-1] D[p] + G_t[p-1] E[p] + R[p] F[p-1]: the rows
        // before this lane's first row come from the lanes 16 below (or, for
        // the sub-block's first row, from the carriers entering it).
        float Gsh[4];
        {
            const float gprev = shfl(dk.G[3], (lane - 16) & 63);
            Gsh[0] = grp == 0 ? 1.0f : gprev;
            Gsh[1] = dk.G[0]; Gsh[2] = dk.G[1]; Gsh[3] = dk.G[2];
        }
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            float E[4], F[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                E[r] = El[m][r] + rrow[r] * pinE[m];
                F[r] = Fl[m][r] + dk.G[r] * sF[m];
            }
            const float wup = shfl(W[m][3], (lane - 16) & 63);
            const float fup = shfl(F[3], (lane - 16) & 63);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float wprev = r > 0 ? W[m][r - 1] : (grp == 0 ? s[m] : wup);
                const float fprev = r > 0 ? F[r - 1] : (grp == 0 ? sF[m] : fup);
                acc[r] += wprev * Dl[m][r] + gp * Gsh[r] * E[r] + Rv[r] * fprev;
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            const float tot = row_sum(acc[r]) * shfl(ds_n, base + 4 * grp + r);
            if (n == 0 && wk.valid && t < wk.t_end) {
                float* dst = dab + t * p.sa_t;
                if (split)
                    atomicAdd(dst, tot);   // exactly two addends onto zero: order-independent
                else
                    *dst = tot;
            }
        }
    }
}

// Zeroes da ([B, T, H] float32 with a's strides) before the virtual heads of
// a head add their channels' shares.
__global__ __launch_bounds__(256) void swr_uni_zero_kernel(float* da, int64_t T, int64_t H, int64_t sa_b,
                                                           int64_t sa_t, int64_t sa_h, int64_t total) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int64_t h = i % H, t = (i / H) % T, b = i / (H * T);
    da[b * sa_b + t * sa_t + h * sa_h] = 0.0f;
}

template <class IO, int CPL, int TW>
hipError_t launch_uni_tw(const Params& p, bool backward, hipStream_t st) {
    constexpr int HW = 8 / TW;
    const dim3 grid((uint32_t)p.nwork), block(TW * HW * 64);
    if (!backward)
        hipLaunchKernelGGL((swr_uni_fwd_kernel<IO, CPL, TW, HW>), grid, block, 0, st, p);
    else if (p.sig_a || p.sig_b)
        hipLaunchKernelGGL((swr_uni_bwd_kernel<IO, CPL, TW, HW, true>), grid, block, 0, st, p);
    else
        hipLaunchKernelGGL((swr_uni_bwd_kernel<IO, CPL, TW, HW, false>), grid, block, 0, st, p);
    return hipGetLastError();
}

template <class IO, int CPL>
hipError_t launch_uni_block(const Params& p, bool backward, hipStream_t st) {
    switch (p.block) {
        case 16: return launch_uni_tw<IO, CPL, 1>(p, backward, st);
        case 32: return launch_uni_tw<IO, CPL, 2>(p, backward, st);
        case 64: return launch_uni_tw<IO, CPL, 4>(p, backward, st);
        case 128: return launch_uni_tw<IO, CPL, 8>(p, backward, st);
        default: return hipErrorInvalidValue;
    }
}

template <class IO>
hipError_t launch_uni_io(const Params& p, int cpl, bool backward, hipStream_t st) {
    switch (cpl) {
        case 1: return launch_uni_block<IO, 1>(p, backward, st);
        case 2: return launch_uni_block<IO, 2>(p, backward, st);
        case 4: return launch_uni_block<IO, 4>(p, backward, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_uniform(const Params& p, int dtype, int cpl, bool backward, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    if (p.nwork <= 0) return hipSuccess;
    if (backward && p.hshift > 0) {
        const int64_t total = p.B * p.T * p.H;
        hipLaunchKernelGGL(swr_uni_zero_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st,
                           p.da, p.T, p.H, p.sa_b, p.sa_t, p.sa_h, total);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return dtype == 1 ? launch_uni_io<IoBf16>(p, cpl, backward, st)
                      : launch_uni_io<IoF32>(p, cpl, backward, st);
}

}  // namespace swr
