// swr_kernels.hip -- gfx950 (CDNA4) kernels of the Sliding Window Recurrence.
//
// Method (Sliding Window Recurrences, Sec. 4.2): the jagged-window operator
// L~ = calL + G Z_b R (the hierarchical decomposition of Sec. 3.2 with the
// carrier transfer operator truncated to T ~ I_b), applied by the Block
// Two-Pass algorithm: a local solve w_t = L_t u_t per block, then the
// rank-one injection x_t = w_t + g_t v_{t-1} of the previous block's last
// local state v_{t-1} = w_{t-1,l}.
//
// How it is mapped onto the MI355X:
//
//  * A wave owns a 16-token sub-block of one (batch, head) and all D channels.
//    Lane (grp, n) = (lane / 16, lane % 16) holds tokens 4*grp .. 4*grp+3 and
//    channels n*CPL .. n*CPL+CPL-1 (CPL = D/16), so each token row is fetched
//    with one contiguous vector load per lane (16 bytes for bf16 at D = 128)
//    and sixteen lanes cover a whole row.
//  * The sub-block's lower-triangular operator L (16 x 16, entries
//    L[i][k] = a_{k+1} ... a_i) is the A operand of a 16x16 MFMA.  Taking the
//    channel slot m of every lane as one MFMA column set makes the MFMA output
//    land in exactly the lanes and registers that loaded its inputs, so no LDS
//    transpose is needed.  L is built with the linear-space construction of
//    Sec. 3.2 (Alg. "Direct (Linear-Space) Materialization"): pre-mask the
//    column with ones, take a cumulative product down the column, zero the
//    strict upper triangle; the column-wise cumulative product is a 16-lane
//    DPP prefix-product scan.  Only products, never ratios: zeros propagate.
//  * bf16 operands: u = b*x is exact in fp32 and splits exactly into two bf16
//    values; L is split the same way; two K=32 MFMAs accumulate
//    (L_hi + L_lo)(u_hi + u_lo) in fp32.  fp32 I/O uses the fp32 MFMA.
//  * Blocks longer than 16 tokens are composed from sub-blocks with the exact
//    hierarchical decomposition (Thm. "Hierarchical Decomposition"): each
//    sub-block's last local row and its decay product go to LDS, and after a
//    single barrier every wave walks the short carrier recurrence of the
//    sub-blocks before it.  Two carriers are kept: the state restarted at the
//    current block's start (its end value is v_t) and the full jagged-window
//    state (restarted at the previous block's start), which is what the
//    outputs use.
//  * A workgroup of NW waves advances over a run of consecutive tokens of one
//    (batch, head), NW*16 tokens per step, carrying the carriers in registers.
//    A run that does not start the sequence first re-reads the block before
//    it (the halo) to recover v; nothing crosses workgroups, so there are no
//    atomics and results are bitwise reproducible.
//  * The backward runs the same sweep.  The gradient of the truncated forward
//    is itself a block two-pass with the carry flowing backwards
//    (du_t = L_t^T dh_t + r_t g_{t+1}^T dh_{t+1}), so each step also looks one
//    step ahead at c, dy and a to obtain the carrier coming from the next
//    block.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swr_device.h"
#include "swr_launch.h"

namespace swr {
namespace {

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------

// A workgroup holds HW heads of one batch entry and TW waves per head: wave
// wv = hw * TW + tw owns sub-block tw of each TW * 16-token step of head hw.
// Several heads per workgroup make each step read neighbouring heads' rows,
// i.e. longer contiguous stretches of the [B, T, H, D] tensors, together.
// At least three waves per SIMD, so that the memory and compute phases of
// several workgroups interleave on a compute unit.
//
// MODE selects what the sweep computes (swr_launch.h): the jagged window
// (kSwr); or, for the exact recurrence, the runs' aggregates -- the end state
// of each run started from zero and the run's decay product -- (kAggregate),
// or the outputs from the exact state entering each run (kExact).  The exact
// modes need no halo and never restart the carrier.  kGrouped is the jagged
// window with b and c shared by groups of p.group heads (their own strides).
// kPaired is the jagged window on heads of D/2 channels taken two at a time
// (work item h = heads 2h, 2h+1): each 16-lane row holds both heads' rows,
// lanes 0-7 the first head's channels and 8-15 the second's, so every lane
// still moves 16-byte slices (and the tiles can be copied through LDS); each
// head has its own decay operator, so the local solve runs once per head
// and every lane keeps its own head's result.
template <class IO, int CPL, int TW, int HW, bool FEAT, int MODE>
__global__ __launch_bounds__(TW * HW * 64, 3) void swr_fwd_kernel(Params p) {
    constexpr bool GG = MODE == kGrouped;
    constexpr bool PAIR = MODE == kPaired;
    constexpr bool SWR = MODE == kSwr || GG || PAIR;
    constexpr int NH = PAIR ? 2 : 1;   // heads per kernel head
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;   // fused featurisation
    constexpr int NW = TW * HW;
    constexpr int D = CPL * SB;
    constexpr int STEP = TW * SB;
    constexpr int ES = IO::ES;
    __shared__ float s_wl[2][NW][D];   // last row of each sub-block's local solve
    __shared__ float s_c[2][NW * NH];  // each sub-block's decay product (per head of a pair)
    // The next step's x, b, c tiles are copied into a wave-private LDS slot
    // while the current step computes (16-byte lane slices only; the slots of
    // a workgroup stay small enough for three workgroups per compute unit).
    using RW = Row<IO, CPL>;
    using LR = LdsRow<RW::BYTES>;
    constexpr bool PREFETCH = RW::BYTES % 16 == 0 && NW * 12 * LR::SLOT_WORDS * 4 <= kFwdPrefetchLds;
    __shared__ __attribute__((aligned(16))) uint32_t s_tile[PREFETCH ? NW : 1][3][4][PREFETCH ? LR::SLOT_WORDS : 1];

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, tw = wv % TW;    // head within the group, sub-block within the step
    const Work wk = decode_work<HW>(p, hw);
    const int l = p.block;
    const int S = l / SB;              // sub-blocks per block (a power of two)
    const int smask = S - 1;
    // First token read: the jagged window re-reads the block before the run.
    const int64_t t_lo = SWR ? max(wk.t_begin - (int64_t)l, (int64_t)0) : wk.t_begin;
    const int64_t halo = SWR && wk.t_begin > 0 ? (l + STEP - 1) / STEP : 0;

    const int hsel = PAIR ? n >> 3 : 0;                  // this lane's head of a pair
    // (first) head of the work item; a head wider than the kernel is split
    // into virtual heads of p.dv channels, starting at channel coff
    const int64_t h0 = PAIR ? 2 * wk.h : wk.h >> p.hshift;
    const int64_t coff = PAIR ? 0 : (wk.h & ((1 << p.hshift) - 1)) * (int64_t)p.dv;
    const bool lane_ok = PAIR || n < p.nlane;            // this lane holds channels of the head
    const int64_t DH = PAIR ? D / NH : p.dh;             // channels of a head (carrier rows)
    const int64_t xo = (wk.b * p.sx_b + h0 * p.sx_h + coff) * ES;
    // b and c: this head's rows, or its group's with shared gates
    const int64_t go = GG ? (wk.b * p.sg_b + (wk.h / p.group) * p.sg_h) * ES : xo;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + go;
    const char* cb = (const char*)p.c + go;
    char* yb = (char*)p.y + xo;
    const char* ab = (const char*)p.a + (wk.b * p.sa_b + h0 * p.sa_h) * ES;
    const int64_t rs = p.sx_t * ES;    // row stride in bytes
    const int64_t gs = GG ? p.sg_t * ES : rs;   // of b and c
    const int64_t as = p.sa_t * ES;
    // this lane's channel slice: n * CPL, or (with a pair) its head's (n & 7) * CPL
    const uint32_t lch = PAIR ? (uint32_t)(hsel * p.sx_h * ES) + (uint32_t)((n & 7) * CPL * ES)
                              : (uint32_t)(n * CPL * ES);
    // (every access of an idle lane is out of range: it reads zeros, stores nothing)
    const uint32_t loff = in_range(lane_ok, (uint32_t)(4 * grp) * (uint32_t)rs + lch);
    const uint32_t goff = GG ? in_range(lane_ok, (uint32_t)(4 * grp) * (uint32_t)gs + (uint32_t)(n * CPL * ES))
                             : loff;
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    // false: only the block carriers (or the run aggregates) are produced
    const bool want_y = MODE != kAggregate && p.y != nullptr;
    float* const vb = MODE != kAggregate && p.carriers ? p.carriers + (wk.b * p.H + h0) * p.nblocks * DH + coff
                                                       : nullptr;
    // this lane's carrier slice within the block's entry, in bytes (idle lanes: out of range)
    const uint32_t vch = in_range(lane_ok, (uint32_t)(PAIR ? hsel * p.nblocks * DH + (n & 7) * CPL : n * CPL) * 4u);
    const __amdgpu_buffer_rsrc_t rv = rsrc(vb);
    const int64_t slot = (wk.b * p.H + wk.h) * p.nruns + wk.run;   // this run's aggregate / carry

    // Carriers at the start of the step: e is the state the outputs use (the
    // jagged-window state, or the exact state), s the block-restarted state.
    float e[CPL], s[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }
    if constexpr (MODE == kExact) {   // the exact state entering the run (stage II's result)
        Row<IoF32, CPL> ci;
        const int64_t j = (wk.b * p.H + wk.h) * p.agg_nruns + wk.t_begin / p.agg_len;
        ci.load(rsrc(p.carry + j * D), (uint32_t)(n * CPL) * 4u);
#pragma unroll
        for (int m = 0; m < CPL; ++m) e[m] = ci.get(m);
    }
    float prod = 1.0f;   // kAggregate: decay product of the run so far

    // Sweep to the end of the run's last block: when the sequence ends inside a
    // block, the step holding that block's last sub-block still computes its
    // carrier (its rows past the end are masked, so it moves no data).
    const int64_t t_stop = ((wk.t_end + l - 1) >> p.lshift) << p.lshift;
    const int64_t t_first = wk.t_begin - halo * STEP;
    // Which rows of which tensor a step reads: x and b from the halo block on,
    // c only where y is written.
    auto ok_xb = [&](int64_t t) { return t >= t_lo && t < wk.t_end; };
    auto ok_c = [&](int64_t t) { return want_y && t >= wk.t_begin && t < wk.t_end; };
    // Copies the x, b, c tiles of the step starting at token t0 into this wave's LDS slot.
    auto prefetch = [&](int64_t t0) {
        const int64_t r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * gs), rc = rsrc(cb + r0 * gs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = loff + (uint32_t)(r * rs), og = goff + (uint32_t)(r * gs);
            LR::template issue<kFwdLoad>(rx, in_range(ok_xb(tr0 + r), o), s_tile[wv][0][r]);
            LR::template issue<kFwdLoad>(rb, in_range(ok_xb(tr0 + r), og), s_tile[wv][1][r]);
            LR::template issue<kFwdLoad>(rc, in_range(ok_c(tr0 + r), og), s_tile[wv][2][r]);
        }
    };
    if constexpr (PREFETCH) {
        if (t_first < t_stop) prefetch(t_first);
    }
    int buf = 0;
    for (int64_t t0 = t_first; t0 < t_stop; t0 += STEP, buf ^= 1) {
        const int64_t r0 = t0 + tw * SB;          // first token of this wave's sub-block (uniform)
        const int64_t tr0 = r0 + 4 * grp;         // first of this lane's four tokens

        // ---- loads -------------------------------------------------------
        const __amdgpu_buffer_rsrc_t ry = rsrc(yb + r0 * rs);
        RW xr[4], br[4], cr[4];
        if constexpr (PREFETCH) {
            // The copies into the slot have landed: an explicit wait rather than
            // the compiler's own tracking of copies into LDS, which was seen to
            // let a read of such a tile go ahead of them in another kernel.
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                LR::read(s_tile[wv][0][r], lane, xr[r].w);
                LR::read(s_tile[wv][1][r], lane, br[r].w);
                LR::read(s_tile[wv][2][r], lane, cr[r].w);
                // (an idle lane's slot holds whatever it held: its values stay in
                // its own MFMA column and channels and are never stored)
                if (!ok_xb(tr0 + r)) { xr[r].zero(); br[r].zero(); }
                if (!ok_c(tr0 + r)) cr[r].zero();
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the slot may be refilled
            if (t0 + STEP < t_stop) prefetch(t0 + STEP);
        } else {
            const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * gs),
                                         rc = rsrc(cb + r0 * gs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = tr0 + r;
                const uint32_t o = loff + (uint32_t)(r * rs), og = goff + (uint32_t)(r * gs);
                xr[r].template load<kFwdLoad>(rx, in_range(ok_xb(t), o));
                br[r].template load<kFwdLoad>(rb, in_range(ok_xb(t), og));
                cr[r].template load<kFwdLoad>(rc, in_range(ok_c(t), og));
            }
        }
        const int64_t ta = r0 + n;
        const bool a_ok = ta >= t_lo && ta < wk.t_end;
        float a_n = load_scalar<IO, kFwdDecay>(rsrc(ab + r0 * as), in_range(a_ok, aoff));
        if (sig_a) a_n = a_ok ? sigmoid(a_n) : 0.0f;
        // Past the end of the sequence the decay is 1 (and u = 0), so the
        // carrier of a partial last block is the state at its last token.
        if (ta >= p.T) a_n = 1.0f;
        float a_n1 = 0.0f;   // the second head's decay of a pair
        if constexpr (PAIR) {
            a_n1 = load_scalar<IO, kFwdDecay>(rsrc(ab + p.sa_h * ES + r0 * as), in_range(a_ok, aoff));
            if (sig_a) a_n1 = a_ok ? sigmoid(a_n1) : 0.0f;
            if (ta >= p.T) a_n1 = 1.0f;
        }

        // ---- local solve W = L U on the matrix cores ---------------------
        const Decay dk = build_decay(a_n, grp, n);
        Decay dk1 = dk;
        if constexpr (PAIR) dk1 = build_decay(a_n1, grp, n);
        f32x4 W[CPL];
        {
            const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
            typename Contract<IO>::A A1 = A;
            if constexpr (PAIR) A1 = Contract<IO>::prep(dk1.L);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);   // pre-gate b*x
                W[m] = Contract<IO>::run(A, u);
                if constexpr (PAIR) {   // the second head's lanes keep its own operator's result
                    const f32x4 W1 = Contract<IO>::run(A1, u);
                    if (hsel) W[m] = W1;
                }
            }
        }
        float Gl[4];   // this lane's head's prefix products at its rows
#pragma unroll
        for (int r = 0; r < 4; ++r) Gl[r] = PAIR && hsel ? dk1.G[r] : dk.G[r];

        // ---- carriers through LDS ------------------------------------------
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[buf][wv][n * CPL + m] = W[m][3];
        }
        if (lane == 63) {
            s_c[buf][wv * NH] = dk.c;
            if constexpr (PAIR) s_c[buf][wv * NH + 1] = dk1.c;
        }
        lds_barrier();

        // A step need not start at a block boundary: phase of its first sub-block.
        const int ph = (int)(t0 >> 4) & smask;
        float ein[CPL], vout[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { ein[m] = 0.f; vout[m] = 0.f; }
#pragma unroll 1
        for (int r = 0; r < TW; ++r) {      // the sub-blocks of this wave's head, in order
            if constexpr (SWR) {
                if (((ph + r) & smask) == 0) {   // a block starts: its carry-in is the previous block's v
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                }
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) ein[m] = e[m];
            }
            const int src = hw * TW + r;
            const float cr_ = s_c[buf][src * NH + hsel];
            if constexpr (MODE == kAggregate) prod *= cr_;
            // One fused multiply-add per carrier step, so that the backward's
            // recomputation of a block's carrier (mode kRecompute) rounds exactly
            // as this walk does.
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float wl = s_wl[buf][src][n * CPL + m];
                e[m] = __builtin_fmaf(cr_, e[m], wl);
                if constexpr (SWR) s[m] = __builtin_fmaf(cr_, s[m], wl);
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) vout[m] = SWR ? s[m] : e[m];
            }
        }
        // The wave holding a block's last sub-block saves that block's carrier
        // for the backward: v_t (the block-restarted end state) for the jagged
        // window, the exact state at the block's end for the exact recurrence.
        if (vb && ((ph + tw) & smask) == smask) {
            const int64_t blk = r0 >> p.lshift;
            const int64_t t_blk = blk << p.lshift;   // first token of the block (it may end past T)
            store_row<IoF32, CPL>(rv, in_range(grp == 0 && t_blk >= wk.t_begin && t_blk < wk.t_end,
                                               (uint32_t)(blk * DH) * 4u + vch), vout);
        }
        if (!want_y) continue;

        // ---- rank-one injection, read-out gate, store ----------------------
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float hv = W[m][r] + Gl[r] * ein[m];
                yv[m] = cr[r].get(m) * hv;
                if (p.residual) yv[m] += xr[r].get(m);
            }
            store_row<IO, CPL, kFwdStore>(ry, in_range(t >= wk.t_begin && t < wk.t_end, loff + (uint32_t)(r * rs)), yv);
        }
    }
    if constexpr (MODE == kAggregate) {   // the run's end state from zero, and its decay product
        store_row<IoF32, CPL>(rsrc(p.agg_v + slot * D), in_range(tw == 0 && grp == 0, (uint32_t)(n * CPL) * 4u), e);
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, prod), rsrc(p.agg_p + slot),
                                              (int)in_range(tw == 0 && lane == 0, 0u), 0, 0);
    }
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------


// Gradient of the truncated forward.  du = L~^T dh with dh = c * dy is itself a
// block two-pass run backwards: du_t = L_t^T dh_t + r_t C_{t+1}, where
// r_t = e_l^T L_t and C_{t+1} = g_{t+1}^T dh_{t+1} comes from the next block.
// The decay gradient of token k (block t) collects, over the channels, the
// state entering step k times the adjoint leaving it, for the two windows
// that contain k:  da_k = sum_mu [ w_{t,k-1} du_k + g_{t,k-1} v_{t-1} D_{t,k} ]
// with w the block-restarted local state, D_t = L_t^T dh_t and v_{t-1} the
// previous block's carrier (w_{t,-1} = 0, g_{t,-1} = 1).  Writing it with the
// jagged-window state H entering row k (H_{-1} = the carrier entering the
// sub-block) and the restarted reverse carrier p:
//     da_k = sum_mu H_{k-1} du_k  -  g_{k-1} r_k sum_mu (e - s)(eps - p)
// where (e, s) / (eps, p) are the forward / reverse carriers entering the
// sub-block; the second sum is one number per sub-block and lane.
//
// Schedule: a workgroup sweeps its run from the last step to the first.  The
// reverse carriers then arrive from the step processed before, and the
// forward carrier entering each step is the previous block's carrier v,
// saved by the forward pass (the paper's "checkpoint only the carrier").
// Only the run's end needs a halo: the first block after the run (c, dy, a)
// gives the reverse carrier entering it.  Nothing is read twice.
//
// MODE kExact gives the gradient of the exact recurrence instead: the adjoint
// entering the run from its end is stage II's result (no halo), the state
// entering each step is the previous block's exact carrier (or the initial
// state), nothing restarts, and the decay gradient is sum_mu H_{k-1} du_k.
//
// MODE kGrouped: the jagged window with b and c shared by groups of heads;
// this head's shares of db and dc go to the float32 workspace p.gws, summed
// over each group afterwards (swr_gate_reduce_kernel).
//
// MODE kRecompute: the jagged window without saved carriers.  The carrier of
// the block before each step is recomputed during the step from that
// block's x, b and a (the rows the next step processes): the same local
// solves and the same walk over its sub-blocks as in the forward, so the
// result equals the saved carrier bit for bit.
template <class IO, int CPL, int TW, int HW, bool FEAT, int MODE>
__global__ __launch_bounds__(TW * HW * 64, 2) void swr_bwd_kernel(Params p) {
    constexpr bool GG = MODE == kGrouped;
    constexpr bool VREC = MODE == kRecompute;
    constexpr bool SWR = MODE == kSwr || GG || VREC;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;   // fused featurisation
    constexpr int NW = TW * HW;
    constexpr int D = CPL * SB;
    constexpr int STEP = TW * SB;      // whole blocks
    constexpr int ES = IO::ES;
    using R_ = Row<IO, CPL>;
    __shared__ float s_wl[2][NW][D];    // last row of each sub-block's local solve L u
    __shared__ float s_df[2][NW][D];    // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_c[2][NW];        // decay product of each sub-block
    // kRecompute: the same two for the sub-blocks of the step before
    __shared__ float s_wlp[VREC ? 2 : 1][VREC ? NW : 1][VREC ? D : 1];
    __shared__ float s_cp[VREC ? 2 : 1][VREC ? NW : 1];

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, tw = wv % TW;    // head within the group, sub-block within the step
    const Work wk = decode_work<HW>(p, hw);
    const int l = p.block;
    const int S = l / SB;              // sub-blocks per block (a power of two)
    const int smask = S - 1;
    const int64_t t_la = min(wk.t_end + (int64_t)l, p.T);   // end (excl.) of the halo block

    // The head of the work item; a head wider than the kernel is split into
    // virtual heads of p.dv channels, starting at channel coff, whose shares of
    // the decay gradient meet in two atomic adds onto a zeroed da (split).
    const int64_t head = wk.h >> p.hshift;
    const int64_t coff = (wk.h & ((1 << p.hshift) - 1)) * (int64_t)p.dv;
    const bool split = p.hshift > 0;
    const bool lane_ok = n < p.nlane;    // this lane holds channels of the head
    // this lane's slice of a carrier row, in bytes (idle lanes: out of range)
    const uint32_t vlane = in_range(lane_ok, (uint32_t)(n * CPL) * 4u);
    const int64_t xo = (wk.b * p.sx_b + head * p.sx_h + coff) * ES;
    // b and c: this head's rows, or its group's with shared gates
    const int64_t go = GG ? (wk.b * p.sg_b + (wk.h / p.group) * p.sg_h) * ES : xo;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + go;
    const char* cb = (const char*)p.c + go;
    const char* dyb = (const char*)p.dy + xo;
    char* dxb = (char*)p.dx + xo;
    // db and dc: this head's float32 shares in the workspace with shared gates
    const int64_t wso = ((wk.b * p.T) * p.H + wk.h) * D;
    char* dbb = GG ? (char*)(p.gws + wso) : (char*)p.db + xo;
    char* dcb = GG ? (char*)(p.gws + p.B * p.T * p.H * D + wso) : (char*)p.dc + xo;
    const int64_t ao = wk.b * p.sa_b + head * p.sa_h;
    const char* ab = (const char*)p.a + ao * ES;
    char* dab = (char*)(p.da + ao);
    const float* vb = p.carriers + (wk.b * p.H + head) * p.nblocks * p.dh + coff;
    const int64_t rs = p.sx_t * ES;
    const int64_t gs = GG ? p.sg_t * ES : rs;        // row stride of b and c
    const int64_t ws = GG ? p.H * D * 4 : rs;         // row stride of db and dc
    const int64_t as = p.sa_t * ES;
    const int64_t das = p.sa_t * 4;
    // (every row access of an idle lane is out of range: it reads zeros, stores nothing)
    const uint32_t loff = in_range(lane_ok, (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES));
    const uint32_t goff = GG ? in_range(lane_ok, (uint32_t)(4 * grp) * (uint32_t)gs + (uint32_t)(n * CPL * ES))
                             : loff;
    const uint32_t woff = GG ? (uint32_t)(4 * grp) * (uint32_t)ws + (uint32_t)(n * CPL * 4) : loff;
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const uint32_t daoff = (uint32_t)(4 * grp) * (uint32_t)das;
    const int base = lane & 48;   // first lane of this 16-lane row

    // Reverse carriers at the end of the step about to be processed: the
    // full adjoint entering from the right (eps) and the one restarted at the
    // end of the current block (pr).
    float eps[CPL], pr[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { eps[m] = 0.f; pr[m] = 0.f; }
    const int64_t seq = wk.b * p.H + wk.h;
    if constexpr (MODE == kExact) {   // the exact adjoint entering the run's end (stage II)
        Row<IoF32, CPL> ci;
        const int64_t j = seq * p.agg_nruns + (wk.t_end - 1) / p.agg_len;   // the run's last aggregate
        ci.load(rsrc(p.carry + j * D), (uint32_t)(n * CPL) * 4u);
#pragma unroll
        for (int m = 0; m < CPL; ++m) eps[m] = ci.get(m);
    }
    int buf = 0;

    // ---- halo: the first block after the run -----------------------------------
    if (SWR && wk.t_end < p.T) {
        const int64_t r0 = wk.t_end + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
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
            if (grp == 0) s_df[buf][wv][n * CPL + m] = a0 * Dn[0];
        }
        const float cq = shfl(row_prefix_prod(a_n), 15);
        if (lane == 0) s_c[buf][wv] = cq;
        lds_barrier();
#pragma unroll 1
        for (int r = TW - 1; r >= 0; --r) {
            if ((r & smask) == smask) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            const int src = hw * TW + r;
            const float c_ = s_c[buf][src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float df = s_df[buf][src][n * CPL + m];
                eps[m] = __builtin_fmaf(c_, eps[m], df);
                pr[m] = __builtin_fmaf(c_, pr[m], df);
            }
        }
        buf ^= 1;
    }

    // A step's inputs: the rows of x, b, c, dy, the decays and the carrier of
    // the block before it.  PF: fetched during the step before (bf16 heads of
    // up to 64 channels, no featurisation; 147 -> 186 VGPRs, which keeps
    // 8-wave groups at one per compute unit and leaves 4-wave groups two of
    // their three, measured faster either way).  The 128-channel kernel has
    // no registers to spare for it.  The fetch is straight-line code (live
    // false: every access out of range, reading zero), so the loads are not
    // waited for where two paths would join.
    constexpr bool PF = CPL <= 4 && IO::ES == 2 && !FEAT;
    struct StepIn {
        R_ x[4], b[4], c[4], dy[4];
        float a;
        float v[CPL];
    };
    auto fetch_step = [&](int64_t kk, bool live, StepIn& in) {
        const int64_t t0 = wk.t_begin + kk * STEP, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * gs), rc = rsrc(cb + r0 * gs),
                                     rdy = rsrc(dyb + r0 * rs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const bool ok = live && tr0 + r < wk.t_end;
            const uint32_t o = in_range(ok, loff + (uint32_t)(r * rs));
            const uint32_t og = GG ? in_range(ok, goff + (uint32_t)(r * gs)) : o;
            in.x[r].template load<kBwdLoad>(rx, o);
            in.b[r].template load<kBwdLoad>(rb, og);
            in.c[r].template load<kBwdLoad>(rc, og);
            in.dy[r].template load<kBwdLoad>(rdy, o);
        }
        in.a = load_scalar<IO, kBwdDecay>(rsrc(ab + r0 * as), in_range(live && r0 + n < wk.t_end, aoff));
        // Carrier of the block before the step (zero before the sequence
        // start, or the initial state for the exact recurrence).
        if constexpr (!VREC) {
            const bool from_h0 = MODE == kExact && t0 == 0;
            const int64_t blk = (t0 >> p.lshift) - 1;
            Row<IoF32, CPL> vr;
            vr.load(rsrc(from_h0 ? (const void*)(p.h0 + seq * D) : (const void*)vb),
                    from_h0 ? in_range(live && p.h0 != nullptr, (uint32_t)(n * CPL) * 4u)
                            : in_range(live && t0 > 0, (uint32_t)(blk * p.dh) * 4u + vlane));
#pragma unroll
            for (int m = 0; m < CPL; ++m) in.v[m] = vr.get(m);
        }
    };

    // kRecompute: the local solves of the step before the one starting at t0
    // (rows of its last block only; none before the sequence), whose last
    // rows and decay products go to LDS for the walk that yields the carrier
    // of the block before t0.  As in the forward sweep.
    auto prev_solve = [&](int64_t t0, int pb) {
        const int64_t r0 = t0 - STEP + tw * SB, tr0 = r0 + 4 * grp;
        const int64_t t_pl = max(t0 - (int64_t)l, (int64_t)0);   // first row needed
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * gs);
        R_ xr[4], br[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const bool ok = tr0 + r >= t_pl;   // (every row lies before t0)
            xr[r].template load<kBwdLoad>(rx, in_range(ok, loff + (uint32_t)(r * rs)));
            br[r].template load<kBwdLoad>(rb, in_range(ok, goff + (uint32_t)(r * gs)));
        }
        const bool a_ok = r0 + n >= t_pl;
        float a_n = load_scalar<IO, kBwdDecay>(rsrc(ab + r0 * as), in_range(a_ok, aoff));
        if (sig_a) a_n = a_ok ? sigmoid(a_n) : 0.0f;
        const Decay dk = build_decay(a_n, grp, n);
        const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            float u[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
            const f32x4 W = Contract<IO>::run(A, u);
            if (grp == 3) s_wlp[pb][wv][n * CPL + m] = W[3];
        }
        if (lane == 63) s_cp[pb][wv] = dk.c;
    };

    const int64_t nsteps = (wk.t_end - wk.t_begin + STEP - 1) / STEP;
    StepIn nxt;
    if constexpr (PF) fetch_step(max(nsteps - 1, (int64_t)0), nsteps > 0, nxt);
    for (int64_t k = nsteps - 1; k >= 0; --k, buf ^= 1) {
        const int64_t t0 = wk.t_begin + k * STEP;      // a block boundary
        const int64_t r0 = t0 + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;

        // ---- loads ---------------------------------------------------------------
        // (kRecompute: the step before is solved first, while few registers are live)
        if constexpr (VREC) prev_solve(t0, buf);
        if constexpr (!PF) fetch_step(k, true, nxt);
        const StepIn in = nxt;
        if constexpr (PF) fetch_step(max(k - 1, (int64_t)0), k > 0, nxt);
        const R_* const xr = in.x;
        const R_* const br = in.b;
        const R_* const dyr = in.dy;
        float dh[4][CPL];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) dh[r][m] = dyr[r].get(m) * in.c[r].get(m);   // dh = dy * c
        float a_n = in.a;
        float ds_n = 1.0f;      // d a / d(input) of token n: 1, or sigma'(z) for a logit z
        if (sig_a) {
            const SigSlope g = sigmoid_slope(a_n);
            ds_n = g.ds;
            a_n = r0 + n < wk.t_end ? g.s : 0.0f;
        }
        // Exact recurrence: past the end of the sequence the decay is 1, so
        // the adjoint entering from the end reaches the last token intact.
        if (MODE == kExact && r0 + n >= p.T) a_n = 1.0f;

        // ---- local solves: W = L (b*x) and Dl = L^T (c*dy) ---------------------------
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
                    d4[q] = dh[q][m];
                }
                W[m] = Contract<IO>::run(A, u);
                Dl[m] = Contract<IO>::run(At, d4);
            }
        }
        const float a0 = shfl(a_n, 0);
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[buf][wv][n * CPL + m] = W[m][3];
        }
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_df[buf][wv][n * CPL + m] = a0 * Dl[m][0];
        }
        if (lane == 63) s_c[buf][wv] = dk.c;
        lds_barrier();

        // ---- forward carriers entering this wave's sub-block ---------------------------
        float ein[CPL], sin_[CPL];
        float vrec[CPL];   // kRecompute: the carrier of the block before the step
        if constexpr (VREC) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) vrec[m] = 0.f;
#pragma unroll 1
            for (int r = 0; r < TW; ++r) {   // the step before starts a block
                if ((r & smask) == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) vrec[m] = 0.f;
                }
                const int src = hw * TW + r;
                const float c_ = s_cp[buf][src];
#pragma unroll
                for (int m = 0; m < CPL; ++m) vrec[m] = __builtin_fmaf(c_, vrec[m], s_wlp[buf][src][n * CPL + m]);
            }
        }
        const float* const vprev = VREC ? vrec : in.v;
        {
            // Exact: e is the exact state (never restarted) and s is unused.
            float e[CPL], s[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) { e[m] = SWR ? 0.f : vprev[m]; s[m] = SWR ? vprev[m] : 0.f; }
#pragma unroll 1
            for (int r = 0; r < tw; ++r) {
                if (SWR && (r & smask) == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                }
                const int src = hw * TW + r;
                const float c_ = s_c[buf][src];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float wl = s_wl[buf][src][n * CPL + m];
                    e[m] = __builtin_fmaf(c_, e[m], wl);
                    if constexpr (SWR) s[m] = __builtin_fmaf(c_, s[m], wl);
                }
            }
            if (SWR && (tw & smask) == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
            }
#pragma unroll
            for (int m = 0; m < CPL; ++m) { ein[m] = e[m]; sin_[m] = s[m]; }
        }

        // ---- reverse carriers: capture at this sub-block, carry to the previous step ---
        float epsin[CPL], kd = 0.f;
#pragma unroll 1
        for (int r = TW - 1; r >= 0; --r) {
            if (SWR && (r & smask) == smask) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    epsin[m] = eps[m];
                    if constexpr (SWR) kd = __builtin_fmaf(ein[m] - sin_[m], eps[m] - pr[m], kd);
                }
            }
            const int src = hw * TW + r;
            const float c_ = s_c[buf][src];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float df = s_df[buf][src][n * CPL + m];
                eps[m] = __builtin_fmaf(c_, eps[m], df);
                if constexpr (SWR) pr[m] = __builtin_fmaf(c_, pr[m], df);
            }
        }

        // ---- gradients -------------------------------------------------------------------
        // H = W + g * e_in: the jagged-window state of each row.
#pragma unroll
        for (int m = 0; m < CPL; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) W[m][r] = __builtin_fmaf(dk.G[r], ein[m], W[m][r]);
        float hup[CPL];   // state entering this lane's first row
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            const float v = shfl(W[m][3], (lane - 16) & 63);
            hup[m] = grp == 0 ? ein[m] : v;
        }
        float Rr[4], Gsh[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Rr[r] = shfl(dk.L[r], base + 15);   // r_q = L[15][.] at this lane's rows
        {
            const float gprev = shfl(dk.G[3], (lane - 16) & 63);      // G[k-1], G[-1] = 1
            Gsh[0] = grp == 0 ? 1.0f : gprev;
            Gsh[1] = dk.G[0]; Gsh[2] = dk.G[1]; Gsh[3] = dk.G[2];
        }
        const __amdgpu_buffer_rsrc_t rdx = rsrc(dxb + r0 * rs), rdb = rsrc(dbb + r0 * ws),
                                     rdc = rsrc(dcb + r0 * ws), rda = rsrc(dab + r0 * das);
        auto out_row = [&](int r, float (&vdx)[CPL], float (&vdb)[CPL], float (&vdc)[CPL], float& tot) {
            float acc = SWR ? -Gsh[r] * Rr[r] * kd : 0.0f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float dyv = dyr[r].get(m);
                vdc[m] = dyv * W[m][r];
                const float du = __builtin_fmaf(Rr[r], epsin[m], Dl[m][r]);   // adjoint of u
                const float zb = FEAT ? fresh(br[r].get(m)) : br[r].get(m);
                const SigSlope g = sig_b ? sigmoid_slope(zb) : SigSlope{zb, 1.0f};
                vdx[m] = g.s * du;
                if (p.residual) vdx[m] += dyv;
                vdb[m] = xr[r].get(m) * du * g.ds;
                acc = __builtin_fmaf(r == 0 ? hup[m] : W[m][r - 1], du, acc);
            }
            tot = row_sum(acc) * shfl(ds_n, base + 4 * grp + r);
        };
        auto store_da = [&](int r, float tot) {
            const int oda = (int)in_range(n == 0 && tr0 + r < wk.t_end, daoff + (uint32_t)(r * das));
            if (split)   // this virtual head's share: two addends onto zero, order-independent
                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(tot, rda, oda, 0, 0);
            else
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, tot), rda, oda, 0, kBwdStore);
        };
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float vdx[CPL], vdb[CPL], vdc[CPL], tot;
            out_row(r, vdx, vdb, vdc, tot);
            const uint32_t o = in_range(t < wk.t_end, loff + (uint32_t)(r * rs));
            store_row<IO, CPL, kBwdStore>(rdx, o, vdx);
            if constexpr (GG) {   // this head's float32 shares, summed over the group later
                const uint32_t ow = in_range(t < wk.t_end, woff + (uint32_t)(r * ws));
                store_row<IoF32, CPL>(rdb, ow, vdb);
                store_row<IoF32, CPL>(rdc, ow, vdc);
            } else {
                store_row<IO, CPL, kBwdStore>(rdb, o, vdb);
                store_row<IO, CPL, kBwdStore>(rdc, o, vdc);
            }
            store_da(r, tot);
        }
    }
}

// Stage I of the exact recurrence's backward: for every run, the adjoint that
// leaves its first token towards the previous one when nothing enters from
// the run's end (the reverse local solve D = L^T dh of the whole run, dh =
// c * dy, scaled by the first token's decay), and the run's decay product.
// Only c, dy and a are read.  Past the end of the sequence the decay is 1.
template <class IO, int CPL, int TW, bool FEAT>
__global__ __launch_bounds__(TW * 64, 2) void swr_bwd_agg_kernel(Params p) {
    const int sig_a = FEAT ? p.sig_a : 0;
    constexpr int D = CPL * SB;
    constexpr int STEP = TW * SB;
    constexpr int ES = IO::ES;
    using R_ = Row<IO, CPL>;
    __shared__ float s_df[2][TW][D];   // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_c[2][TW];       // decay product of each sub-block

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const Work wk = decode_work<1>(p, 0);
    const int64_t xo = (wk.b * p.sx_b + wk.h * p.sx_h) * ES;
    const char* cb = (const char*)p.c + xo;
    const char* dyb = (const char*)p.dy + xo;
    const char* ab = (const char*)p.a + (wk.b * p.sa_b + wk.h * p.sa_h) * ES;
    const int64_t rs = p.sx_t * ES;
    const int64_t as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const int64_t slot = (wk.b * p.H + wk.h) * p.nruns + wk.run;

    float eps[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) eps[m] = 0.f;
    float prod = 1.0f;
    int buf = 0;
    const int64_t nsteps = (wk.t_end - wk.t_begin + STEP - 1) / STEP;
    for (int64_t k = nsteps - 1; k >= 0; --k, buf ^= 1) {
        const int64_t r0 = wk.t_begin + k * STEP + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs);
        R_ cr[4], dyr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(tr0 + r < wk.t_end, loff + (uint32_t)(r * rs));
            cr[r].template load<kAggLoad>(rc, o);
            dyr[r].template load<kAggLoad>(rdy, o);
        }
        float a_n = load_scalar<IO, kAggLoad>(rsrc(ab + r0 * as), in_range(r0 + n < wk.t_end, aoff));
        if (sig_a) a_n = sigmoid(a_n);
        if (r0 + n >= p.T) a_n = 1.0f;
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
            const float c_ = s_c[buf][r];
            prod *= c_;
#pragma unroll
            for (int m = 0; m < CPL; ++m) eps[m] = c_ * eps[m] + s_df[buf][r][n * CPL + m];
        }
    }
    store_row<IoF32, CPL>(rsrc(p.agg_v + slot * D), in_range(tw == 0 && grp == 0, (uint32_t)(n * CPL) * 4u), eps);
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, prod), rsrc(p.agg_p + slot),
                                          (int)in_range(tw == 0 && lane == 0, 0u), 0, 0);
}

// Stage II of the exact recurrence: the carrier recurrence over the runs of
// one sequence (Alg. "Hierarchical Block Parallel Inference", global carrier
// solve, here at run granularity), one thread per (sequence, channel).  The
// runs' aggregates are loaded eight at a time ahead of the dependent chain.
__global__ __launch_bounds__(256) void swr_scan_kernel(ScanParams q) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= q.seqs * q.D) return;
    const int64_t seq = idx / q.D, ch = idx - seq * q.D;
    const float* v = q.agg_v + seq * q.nruns * q.D + ch;
    const float* pp = q.p_per_channel ? q.agg_p + seq * q.nruns * q.D + ch : q.agg_p + seq * q.nruns;
    const int64_t pstride = q.p_per_channel ? q.D : 1;
    float* cy = q.carry + seq * q.nruns * q.D + ch;
    float S = q.init ? q.init[idx] : 0.0f;
    constexpr int G = 8;
    for (int64_t r0 = 0; r0 < q.nruns; r0 += G) {
        float vv[G], pv[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int64_t j = r0 + g;
            const int64_t r = q.reverse ? q.nruns - 1 - j : j;
            vv[g] = j < q.nruns ? v[r * q.D] : 0.0f;
            pv[g] = j < q.nruns ? pp[r * pstride] : 1.0f;
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int64_t j = r0 + g;
            if (j < q.nruns) {
                const int64_t r = q.reverse ? q.nruns - 1 - j : j;
                cy[r * q.D] = S;
                S = pv[g] * S + vv[g];
            }
        }
    }
    if (q.fin) q.fin[idx] = S;
}

// ---------------------------------------------------------------------------
// Plain global accesses (per-lane 64-bit addresses)
// ---------------------------------------------------------------------------
//
// The buffer accesses above take their base address from a wave-uniform
// resource; where every lane addresses a different (batch, head), as in the
// decoding kernels below, a per-lane base would make the compiler loop over
// the lanes' distinct resources.  These load and store a lane's row slice
// through an ordinary pointer instead.

template <class IO, int CPL>
__device__ inline void gload(Row<IO, CPL>& r, const void* p) {
    constexpr int BYTES = Row<IO, CPL>::BYTES;
    if constexpr (BYTES == 2) {
        r.w[0] = *(const uint16_t*)p;
    } else if constexpr (BYTES == 4) {
        r.w[0] = *(const uint32_t*)p;
    } else if constexpr (BYTES == 8) {
        const uint2 v = *(const uint2*)p;
        r.w[0] = v.x; r.w[1] = v.y;
    } else {
#pragma unroll
        for (int i = 0; i < BYTES / 16; ++i) {
            const uint4 v = ((const uint4*)p)[i];
            r.w[4 * i + 0] = v.x; r.w[4 * i + 1] = v.y; r.w[4 * i + 2] = v.z; r.w[4 * i + 3] = v.w;
        }
    }
}

template <class IO, int CPL>
__device__ inline void gstore(void* p, const float (&v)[CPL]) {
    constexpr int BYTES = CPL * IO::ES;
    uint32_t w[BYTES >= 4 ? BYTES / 4 : 1];
    if constexpr (IO::ES == 2) {
        if constexpr (CPL == 1) {
            *(uint16_t*)p = (uint16_t)IoBf16::from_f32(v[0]);
            return;
        } else {
#pragma unroll
            for (int i = 0; i < CPL / 2; ++i)
                w[i] = IoBf16::from_f32(v[2 * i]) | (IoBf16::from_f32(v[2 * i + 1]) << 16);
        }
    } else {
#pragma unroll
        for (int i = 0; i < CPL; ++i) w[i] = __builtin_bit_cast(uint32_t, v[i]);
    }
    if constexpr (BYTES == 4) {
        *(uint32_t*)p = w[0];
    } else if constexpr (BYTES == 8) {
        *(uint2*)p = uint2{w[0], w[1]};
    } else if constexpr (BYTES >= 16) {
#pragma unroll
        for (int i = 0; i < BYTES / 16; ++i) ((uint4*)p)[i] = uint4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
    }
}

template <class IO>
__device__ inline float gload_scalar(const void* p) {
    if constexpr (IO::ES == 2)
        return IoBf16::to_f32(*(const uint16_t*)p);
    else
        return *(const float*)p;
}

// ---------------------------------------------------------------------------
// Recurrent steps (decoding)
// ---------------------------------------------------------------------------
//
// One thread per (batch, head) and 16th of the channels (the lane slice of the
// block kernels, so the same alignment rules hold); the tokens of a call are
// taken in order.  The jagged window is carried as two states per channel
// (Sec. 4.2's window as a recurrence): e, restarted at the start of the
// previous block, which the outputs read, and s, restarted at the start of
// the current block; when a block starts, e takes s and s restarts from zero.
// The exact recurrence carries h alone.  Work per token is a few flops per
// channel: a launch of a handful of tokens is bound by latency, not by HBM.
// Gates shared by groups of heads: sums each group's float32 shares of db and
// dc, which the kGrouped backward left in p.gws ([2][B][T][H][D]), over the
// group's heads in head order (so the result does not depend on scheduling)
// and stores db and dc ([B, T, H / group, D], strides sg_*) in the I/O dtype.
// One thread per (batch, token, group, 16th of the channels).
template <class IO, int CPL>
__global__ __launch_bounds__(256) void swr_gate_reduce_kernel(Params p) {
    constexpr int D = CPL * SB;
    const int64_t G = p.H / p.group;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= p.B * p.T * G * 16) return;
    const int n = (int)(i & 15);
    const int64_t rest = i >> 4;
    const int64_t g = rest % G, t = (rest / G) % p.T, b = rest / (G * p.T);
    const float* src = p.gws + ((b * p.T + t) * p.H + g * p.group) * D + n * CPL;
    const int64_t half = p.B * p.T * p.H * D;
    float vb[CPL], vc[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { vb[m] = 0.f; vc[m] = 0.f; }
    for (int64_t j = 0; j < p.group; ++j) {
        Row<IoF32, CPL> rb, rc;
        gload<IoF32, CPL>(rb, src + j * D);
        gload<IoF32, CPL>(rc, src + half + j * D);
#pragma unroll
        for (int m = 0; m < CPL; ++m) { vb[m] += rb.get(m); vc[m] += rc.get(m); }
    }
    const int64_t o = (b * p.sg_b + t * p.sg_t + g * p.sg_h + n * CPL) * IO::ES;
    gstore<IO, CPL>((char*)p.db + o, vb);
    gstore<IO, CPL>((char*)p.dc + o, vc);
}

template <class IO, int CPL, bool EXACT, bool PC, bool FEAT>
__global__ __launch_bounds__(256) void swr_step_kernel(StepParams q) {
    constexpr int D = CPL * SB;
    constexpr int ES = IO::ES;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= q.B * q.H * 16) return;   // no barriers below: idle threads may leave
    const int sig_a = FEAT ? q.sig_a : 0, sig_b = FEAT ? q.sig_b : 0;
    const int64_t seq = idx >> 4;
    const int n = (int)(idx & 15);
    const int64_t bb = seq / q.H, hh = seq - bb * q.H;
    const int64_t xo = (bb * q.sx_b + hh * q.sx_h) * ES + n * CPL * ES;   // this thread's slice, token 0
    const int64_t ao = PC ? xo : (bb * q.sa_b + hh * q.sa_h) * ES;
    const int64_t rs = q.sx_t * ES, as = PC ? rs : q.sa_t * ES;
    float* st = q.state + seq * (EXACT ? D : 2 * D) + n * CPL;

    float e[CPL], s[CPL];
    {
        Row<IoF32, CPL> re, rs_;
        gload(re, st);
        if constexpr (!EXACT) gload(rs_, st + D);
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            e[m] = re.get(m);
            s[m] = EXACT ? 0.f : rs_.get(m);
        }
    }
    for (int64_t k = 0; k < q.K; ++k) {
        const int64_t t = q.t0 + k;
        Row<IO, CPL> xr, br, cr, ar;
        gload(xr, (const char*)q.x + xo + k * rs);
        gload(br, (const char*)q.b + xo + k * rs);
        gload(cr, (const char*)q.c + xo + k * rs);
        float av[CPL];
        if constexpr (PC) {
            gload(ar, (const char*)q.a + ao + k * as);
#pragma unroll
            for (int m = 0; m < CPL; ++m) av[m] = ar.get(m);
        } else {
            const float a1 = gload_scalar<IO>((const char*)q.a + ao + k * as);
#pragma unroll
            for (int m = 0; m < CPL; ++m) av[m] = a1;
        }
        const bool restart = !EXACT && (t & (q.block - 1)) == 0;   // a block starts at t
        float yv[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            const float a_ = sig_a ? sigmoid(av[m]) : av[m];
            const float u = xr.get(m) * pregate(br.get(m), sig_b);
            if (restart) { e[m] = s[m]; s[m] = 0.f; }
            e[m] = a_ * e[m] + u;
            if constexpr (!EXACT) s[m] = a_ * s[m] + u;
            yv[m] = cr.get(m) * e[m];
            if (q.residual) yv[m] += xr.get(m);
        }
        gstore<IO, CPL>((char*)q.y + xo + k * rs, yv);
    }
    gstore<IoF32, CPL>(st, e);
    if constexpr (!EXACT) gstore<IoF32, CPL>(st + D, s);
}

// The jagged window's state after tokens 0 .. T-1, from the forward's block
// carriers: s is the carrier of the last (possibly partial) block tau, whose
// window restarts at that block's start; e restarts one block earlier, so it
// adds the previous block's carrier carried through the last block's decays,
// e = s + (a_{tau l} ... a_{T-1}) v_{tau-1}.
template <class IO, int CPL, bool PC, bool FEAT>
__global__ __launch_bounds__(256) void swr_state_kernel(StateParams q) {
    constexpr int D = CPL * SB;
    constexpr int ES = IO::ES;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= q.B * q.H * 16) return;
    const int sig_a = FEAT ? q.sig_a : 0;
    const int64_t seq = idx >> 4;
    const int n = (int)(idx & 15);
    const int64_t bb = seq / q.H, hh = seq - bb * q.H;
    float e[CPL], s[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }
    if (q.T > 0) {
        const int64_t tau = (q.T - 1) >> q.lshift, t_blk = tau << q.lshift;
        const float* vb = q.carriers + seq * q.nblocks * D + n * CPL;
        Row<IoF32, CPL> rv, rp;
        gload(rv, vb + tau * D);
        if (tau > 0)
            gload(rp, vb + (tau - 1) * D);
        else
            rp.zero();
        const char* ab = (const char*)q.a + (bb * q.sa_b + hh * q.sa_h) * ES + (PC ? n * CPL * ES : 0);
        const int64_t as = q.sa_t * ES;
        float G[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) G[m] = 1.f;
        for (int64_t t = t_blk; t < q.T; ++t) {
            if constexpr (PC) {
                Row<IO, CPL> ar;
                gload(ar, ab + t * as);
#pragma unroll
                for (int m = 0; m < CPL; ++m) G[m] *= sig_a ? sigmoid(ar.get(m)) : ar.get(m);
            } else {
                const float a1 = gload_scalar<IO>(ab + t * as);
                const float a_ = sig_a ? sigmoid(a1) : a1;
#pragma unroll
                for (int m = 0; m < CPL; ++m) G[m] *= a_;
            }
        }
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            s[m] = rv.get(m);
            e[m] = s[m] + G[m] * rp.get(m);
        }
    }
    float* st = q.state + seq * 2 * D + n * CPL;
    gstore<IoF32, CPL>(st, e);
    gstore<IoF32, CPL>(st + D, s);
}

// ---------------------------------------------------------------------------
// Per-channel decay
// ---------------------------------------------------------------------------
//
// With a decay a_{k,mu} per token and channel, every channel is its own scalar
// recurrence: the sub-block operator differs from channel to channel, so the
// local solve is no longer one matrix product shared by the channels.  It is
// a first-order linear scan instead, done per lane and channel: the lane's
// four tokens in order, then a doubling scan over the four 16-lane rows
// (tokens 0-3, 4-7, 8-11, 12-15) of the wave.  Everything else -- sub-blocks
// composed through LDS, block carriers, runs, halos, the reverse sweep of the
// backward -- is the scheme of the shared-decay kernels with each decay
// product kept per channel.  Since no quantity couples channels any more, a
// head of D = 128 channels is processed as two independent halves ("virtual
// heads" of 64 channels), which keeps the per-channel products in registers.

// Reverse local solve of one sub-block, per channel:  D_k = dh_k + a_{k+1} D_{k+1}
// (D_16 = 0), i.e. D = L^T dh, and R_k = a_{k+1} ... a_15 (R_15 = 1).  It runs
// on E_k = a_k D_k, the adjoint leaving token k towards k-1, so that each row
// uses only its own decays: E_k = a_k (dh_k + E_{k+1}).  E is carried
// backwards through a stretch by e -> Q e + E_loc with Q the stretch's decay
// product.
template <int CPL>
__device__ inline void chan_scan_rev(const float (&a)[4][CPL], const float (&dh)[4][CPL],
                                     float (&Dv)[4][CPL], float (&R)[4][CPL], int grp, int lane) {
#pragma unroll
    for (int m = 0; m < CPL; ++m) {
        // In-lane pass with nothing entering from the next row.
        Dv[3][m] = dh[3][m];
        R[3][m] = 1.0f;
#pragma unroll
        for (int r = 2; r >= 0; --r) {
            Dv[r][m] = dh[r][m] + a[r + 1][m] * Dv[r + 1][m];
            R[r][m] = a[r + 1][m] * R[r + 1][m];
        }
        // Row totals: Q = a_{4g} ... a_{4g+3}, E_loc = a_{4g} D_loc(4g).
        float tq = a[0][m] * R[0][m], te = a[0][m] * Dv[0][m];
        // Inclusive scan over rows grp..3.
        float pq = shfl(tq, (lane + 16) & 63), pe = shfl(te, (lane + 16) & 63);
        if (grp <= 2) { te = tq * pe + te; tq = tq * pq; }
        pq = shfl(tq, (lane + 32) & 63); pe = shfl(te, (lane + 32) & 63);
        if (grp <= 1) { te = tq * pe + te; tq = tq * pq; }
        // Exclusive: E entering the row from the next one, and the decay
        // product of the tokens after the row.
        pq = shfl(tq, (lane + 16) & 63); pe = shfl(te, (lane + 16) & 63);
        const float lam = grp <= 2 ? pe : 0.0f, qin = grp <= 2 ? pq : 1.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            Dv[r][m] += R[r][m] * lam;
            R[r][m] *= qin;
        }
    }
}

// Per-channel forward.  Same workgroup shape and sweep as swr_fwd_kernel;
// wk.h is a virtual head: head wk.h >> hshift, channel half wk.h & (2^hshift - 1).
// MODE as for swr_fwd_kernel; the exact modes keep a decay product per
// channel for each run.
template <class IO, int CPL, int TW, int HW, bool FEAT, int MODE, int PK>
__global__ __launch_bounds__(TW * HW * 64, 3) void swr_fwd_pc_kernel(Params p) {
    constexpr bool SWR = MODE == kSwr;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;   // fused featurisation
    constexpr int NW = TW * HW;
    constexpr int D = CPL * SB;        // channels of a virtual head
    constexpr int STEP = TW * SB;
    constexpr int ES = IO::ES;
    using RW = Row<IO, CPL>;
    __shared__ float s_wl[2][NW][D];   // last row of each sub-block's local solve
    __shared__ float s_cc[2][NW][D];   // each sub-block's decay product, per channel

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, tw = wv % TW;
    const Work wk = decode_work<HW>(p, hw);
    const Geo<PK, CPL> geo(wk.h, p, n);
    const int l = p.block;
    const int smask = l / SB - 1;
    const int64_t t_lo = SWR ? max(wk.t_begin - (int64_t)l, (int64_t)0) : wk.t_begin;
    const int64_t halo = SWR && wk.t_begin > 0 ? (l + STEP - 1) / STEP : 0;

    const int64_t xo = (wk.b * p.sx_b + geo.head * p.sx_h + geo.coff) * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    // per-channel decay: rows like x; packed heads: one decay per token and real head
    const char* ab = PK > 1 ? (const char*)p.a + (wk.b * p.sa_b + geo.head * p.sa_h) * ES : (const char*)p.a + xo;
    char* yb = (char*)p.y + xo;
    const int64_t rs = p.sx_t * ES;
    const int64_t as = PK > 1 ? p.sa_t * ES : rs;
    const uint32_t loff = in_range(geo.ok, (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES));
    const uint32_t aoffp = (uint32_t)(4 * grp) * (uint32_t)as + (uint32_t)(geo.lh * p.sa_h * ES);
    const bool want_y = MODE != kAggregate && p.y != nullptr;
    const int64_t hb = wk.b * p.H + geo.head;   // first real (batch, head) of the virtual head
    float* const vb = MODE != kAggregate && p.carriers ? p.carriers + hb * p.nblocks * geo.Dr : nullptr;
    const __amdgpu_buffer_rsrc_t rv = rsrc(vb);

    float e[CPL], s[CPL], prod[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; prod[m] = 1.f; }
    if constexpr (MODE == kExact) {
        Row<IoF32, CPL> ci;
        ci.load(rsrc(p.carry + hb * p.agg_nruns * geo.Dr), geo.off(p.agg_nruns, wk.t_begin / p.agg_len) * 4u);
#pragma unroll
        for (int m = 0; m < CPL; ++m) e[m] = ci.get(m);
    }
    const int64_t t_stop = ((wk.t_end + l - 1) >> p.lshift) << p.lshift;
    const int64_t t_first = wk.t_begin - halo * STEP;
    int buf = 0;
    for (int64_t t0 = t_first; t0 < t_stop; t0 += STEP, buf ^= 1) {
        const int64_t r0 = t0 + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs),
                                     rc = rsrc(cb + r0 * rs), ra = rsrc(ab + r0 * as);
        RW xr[4], br[4], cr[4], ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            const uint32_t o = loff + (uint32_t)(r * rs);
            const bool in_xb = t >= t_lo && t < wk.t_end;
            xr[r].template load<kFwdLoad>(rx, in_range(in_xb, o));
            br[r].template load<kFwdLoad>(rb, in_range(in_xb, o));
            if constexpr (PK == 1) ar[r].template load<kFwdLoad>(ra, in_range(in_xb, o));
            cr[r].template load<kFwdLoad>(rc, in_range(want_y && t >= wk.t_begin && t < wk.t_end, o));
        }
        float av[4][CPL], u[4][CPL], W[4][CPL], G[4][CPL];
        if constexpr (PK > 1) {
            float az[4];
            decay_rows_packed<IO, CPL, kFwdDecay>(ra, aoffp, (uint32_t)as, tr0, t_lo, wk.t_end, p.T, sig_a, az, av);
        } else {
            decay_rows<IO, CPL>(ar, tr0, t_lo, wk.t_end, p.T, sig_a, av);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) u[r][m] = xr[r].get(m) * pregate(br[r].get(m), sig_b);
        chan_scan_fwd<CPL>(av, u, W, G, grp, lane);

        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_wl[buf][wv][n * CPL + m] = W[3][m];
                s_cc[buf][wv][n * CPL + m] = G[3][m];
            }
        }
        lds_barrier();

        const int ph = (int)(t0 >> 4) & smask;
        float ein[CPL], vout[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { ein[m] = 0.f; vout[m] = 0.f; }
#pragma unroll 1
        for (int r = 0; r < TW; ++r) {
            if (SWR && ((ph + r) & smask) == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) ein[m] = e[m];
            }
            const int src = hw * TW + r;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float c_ = s_cc[buf][src][n * CPL + m];
                const float wl = s_wl[buf][src][n * CPL + m];
                e[m] = __builtin_fmaf(c_, e[m], wl);
                if constexpr (SWR) s[m] = __builtin_fmaf(c_, s[m], wl);
                if constexpr (MODE == kAggregate) prod[m] *= c_;
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) vout[m] = SWR ? s[m] : e[m];
            }
        }
        if (vb && ((ph + tw) & smask) == smask) {
            const int64_t blk = r0 >> p.lshift;
            const int64_t t_blk = blk << p.lshift;
            store_row<IoF32, CPL>(rv, in_range(grp == 0 && geo.ok && t_blk >= wk.t_begin && t_blk < wk.t_end,
                                               geo.off(p.nblocks, blk) * 4u), vout);
        }
        if (!want_y) continue;

        const __amdgpu_buffer_rsrc_t ry = rsrc(yb + r0 * rs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                yv[m] = cr[r].get(m) * (W[r][m] + G[r][m] * ein[m]);
                if (p.residual) yv[m] += xr[r].get(m);
            }
            store_row<IO, CPL, kFwdStore>(ry, in_range(t >= wk.t_begin && t < wk.t_end, loff + (uint32_t)(r * rs)), yv);
        }
    }
    if constexpr (MODE == kAggregate) {   // the run's end state from zero and decay products
        const uint32_t o = in_range(tw == 0 && grp == 0, geo.off(p.nruns, wk.run) * 4u);
        store_row<IoF32, CPL>(rsrc(p.agg_v + hb * p.nruns * geo.Dr), o, e);
        store_row<IoF32, CPL>(rsrc(p.agg_p + hb * p.nruns * geo.Dr), o, prod);
    }
}

// Per-channel backward: the reverse sweep of swr_bwd_kernel with per-channel
// decay products.  The decay gradient keeps its closed form per channel,
//     da_{k,mu} = H_{k-1,mu} du_{k,mu} - g_{k-1,mu} r_{k,mu} (e - s)_mu (eps - p)_mu,
// and is stored per channel (no sum over the head's channels).
// MODE kExact: the gradient of the exact recurrence, as in swr_bwd_kernel.
// MODE kRecompute: without saved carriers, as in swr_bwd_kernel.
template <class IO, int CPL, int TW, int HW, bool FEAT, int MODE, int PK>
__global__ __launch_bounds__(TW * HW * 64, 2) void swr_bwd_pc_kernel(Params p) {
    constexpr bool VREC = MODE == kRecompute;
    constexpr bool SWR = MODE == kSwr || VREC;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;   // fused featurisation
    constexpr int NW = TW * HW;
    constexpr int D = CPL * SB;
    constexpr int STEP = TW * SB;      // whole blocks
    constexpr int ES = IO::ES;
    using R_ = Row<IO, CPL>;
    __shared__ float s_wl[2][NW][D];    // last row of each sub-block's local solve L u
    __shared__ float s_df[2][NW][D];    // E_0 = a_0 D_0 of each sub-block's L^T dh
    __shared__ float s_cc[2][NW][D];    // decay product of each sub-block, per channel
    // kRecompute: the same two for the sub-blocks of the step before
    __shared__ float s_wlp[VREC ? 2 : 1][VREC ? NW : 1][VREC ? D : 1];
    __shared__ float s_ccp[VREC ? 2 : 1][VREC ? NW : 1][VREC ? D : 1];

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const int hw = wv / TW, tw = wv % TW;
    const Work wk = decode_work<HW>(p, hw);
    const Geo<PK, CPL> geo(wk.h, p, n);
    const int l = p.block;
    const int smask = l / SB - 1;
    const int64_t t_la = min(wk.t_end + (int64_t)l, p.T);

    const int64_t xe = wk.b * p.sx_b + geo.head * p.sx_h + geo.coff;   // element offset
    const int64_t xo = xe * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    const char* dyb = (const char*)p.dy + xo;
    char* dxb = (char*)p.dx + xo;
    char* dbb = (char*)p.db + xo;
    char* dcb = (char*)p.dc + xo;
    // per-channel decay: a and da are rows like x; packed heads: one decay per
    // token and real head (da float32 with a's strides)
    const int64_t ae = PK > 1 ? wk.b * p.sa_b + geo.head * p.sa_h : xe;
    const char* ab = (const char*)p.a + ae * ES;
    char* dab = (char*)(p.da + ae);
    const int64_t hb = wk.b * p.H + geo.head;   // first real (batch, head) of the virtual head
    const float* vb = p.carriers + hb * p.nblocks * geo.Dr;
    const int64_t rs = p.sx_t * ES;
    const int64_t as = PK > 1 ? p.sa_t * ES : rs;
    const int64_t das = PK > 1 ? p.sa_t * 4 : p.sx_t * 4;
    const uint32_t loff = in_range(geo.ok, (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES));
    const uint32_t aoffp = (uint32_t)(4 * grp) * (uint32_t)as + (uint32_t)(geo.lh * p.sa_h * ES);
    const uint32_t daoff = PK > 1 ? (uint32_t)(4 * grp) * (uint32_t)das + (uint32_t)(geo.lh * p.sa_h * 4)
                                  : in_range(geo.ok, (uint32_t)(4 * grp) * (uint32_t)das + (uint32_t)(n * CPL * 4));

    float eps[CPL], pr[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { eps[m] = 0.f; pr[m] = 0.f; }
    if constexpr (MODE == kExact) {   // the exact adjoint entering the run's end (stage II)
        Row<IoF32, CPL> ci;
        // the run's last aggregate
        ci.load(rsrc(p.carry + hb * p.agg_nruns * geo.Dr), geo.off(p.agg_nruns, (wk.t_end - 1) / p.agg_len) * 4u);
#pragma unroll
        for (int m = 0; m < CPL; ++m) eps[m] = ci.get(m);
    }
    int buf = 0;

    // ---- halo: the first block after the run -----------------------------------
    if (SWR && wk.t_end < p.T) {
        const int64_t r0 = wk.t_end + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs),
                                     ra = rsrc(ab + r0 * as);
        R_ cr[4], dyr[4], ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(tr0 + r < t_la, loff + (uint32_t)(r * rs));
            cr[r].template load<kBwdLoad>(rc, o);
            dyr[r].template load<kBwdLoad>(rdy, o);
            if constexpr (PK == 1) ar[r].template load<kBwdLoad>(ra, o);
        }
        float av[4][CPL], dh[4][CPL], Dv[4][CPL], R[4][CPL];
        if constexpr (PK > 1) {   // (past T the 1s meet dh = 0)
            float az[4];
            decay_rows_packed<IO, CPL, kBwdDecay>(ra, aoffp, (uint32_t)as, tr0, wk.t_end, t_la, p.T, sig_a, az, av);
        } else {
            decay_rows<IO, CPL>(ar, tr0, wk.t_end, t_la, p.T, sig_a, av);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) dh[r][m] = dyr[r].get(m) * cr[r].get(m);
        chan_scan_rev<CPL>(av, dh, Dv, R, grp, lane);
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_df[buf][wv][n * CPL + m] = av[0][m] * Dv[0][m];
                s_cc[buf][wv][n * CPL + m] = av[0][m] * R[0][m];   // a_0 ... a_15
            }
        }
        lds_barrier();
#pragma unroll 1
        for (int r = TW - 1; r >= 0; --r) {
            if ((r & smask) == smask) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            const int src = hw * TW + r;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float c_ = s_cc[buf][src][n * CPL + m];
                const float df = s_df[buf][src][n * CPL + m];
                eps[m] = __builtin_fmaf(c_, eps[m], df);
                pr[m] = __builtin_fmaf(c_, pr[m], df);
            }
        }
        buf ^= 1;
    }

    // A step's inputs: the rows of x, b, c, dy (and of a, one decay per
    // channel) and the carrier of the block before it.  PF: fetched during
    // the step before (bf16, one decay per channel, no featurisation: the
    // float32 kernels would spill, the featurised ones measured no faster).
    // The fetch is straight-line code (live false: every access out of
    // range, reading zero), so the loads are not waited for where two paths
    // would join.
    constexpr bool PF = PK == 1 && IO::ES == 2 && !FEAT;
    struct StepIn {
        R_ x[4], b[4], c[4], dy[4], a[4];
        float v[CPL];
    };
    auto fetch_step = [&](int64_t kk, bool live, StepIn& in) {
        const int64_t t0 = wk.t_begin + kk * STEP, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs), rc = rsrc(cb + r0 * rs),
                                     rdy = rsrc(dyb + r0 * rs), ra = rsrc(ab + r0 * as);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(live && tr0 + r < wk.t_end, loff + (uint32_t)(r * rs));
            in.x[r].template load<kBwdLoad>(rx, o);
            in.b[r].template load<kBwdLoad>(rb, o);
            in.c[r].template load<kBwdLoad>(rc, o);
            in.dy[r].template load<kBwdLoad>(rdy, o);
            if constexpr (PK == 1) in.a[r].template load<kBwdLoad>(ra, o);
        }
        // the carrier: the initial state for the exact recurrence's first block
        if constexpr (!VREC) {
            const bool from_h0 = MODE == kExact && t0 == 0;
            const int64_t blk = (t0 >> p.lshift) - 1;
            Row<IoF32, CPL> vr;
            vr.load(rsrc(from_h0 ? p.h0 + hb * geo.Dr : vb),
                    from_h0 ? in_range(live && p.h0 != nullptr, geo.off(1, 0) * 4u)
                            : in_range(live && t0 > 0 && geo.ok, geo.off(p.nblocks, blk) * 4u));
#pragma unroll
            for (int m = 0; m < CPL; ++m) in.v[m] = vr.get(m);
        }
    };

    // kRecompute: the local solves of the step before the one starting at t0
    // (rows of its last block only; none before the sequence), whose last
    // rows and decay products go to LDS for the walk that yields the carrier
    // of the block before t0.  As in the forward sweep.
    auto prev_solve = [&](int64_t t0, int pb) {
        const int64_t r0 = t0 - STEP + tw * SB, tr0 = r0 + 4 * grp;
        const int64_t t_pl = max(t0 - (int64_t)l, (int64_t)0);   // first row needed
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs), ra = rsrc(ab + r0 * as);
        R_ xr[4], br[4], ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(tr0 + r >= t_pl, loff + (uint32_t)(r * rs));   // (all before t0)
            xr[r].template load<kBwdLoad>(rx, o);
            br[r].template load<kBwdLoad>(rb, o);
            if constexpr (PK == 1) ar[r].template load<kBwdLoad>(ra, o);
        }
        float av[4][CPL], u[4][CPL], W[4][CPL], G[4][CPL];
        if constexpr (PK > 1) {
            float az[4];
            decay_rows_packed<IO, CPL, kBwdDecay>(ra, aoffp, (uint32_t)as, tr0, t_pl, t0, p.T, sig_a, az, av);
        } else {
            decay_rows<IO, CPL>(ar, tr0, t_pl, t0, p.T, sig_a, av);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) u[r][m] = xr[r].get(m) * pregate(br[r].get(m), sig_b);
        chan_scan_fwd<CPL>(av, u, W, G, grp, lane);
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_wlp[pb][wv][n * CPL + m] = W[3][m];
                s_ccp[pb][wv][n * CPL + m] = G[3][m];
            }
        }
    };

    const int64_t nsteps = (wk.t_end - wk.t_begin + STEP - 1) / STEP;
    StepIn nxt;
    if constexpr (PF) fetch_step(max(nsteps - 1, (int64_t)0), nsteps > 0, nxt);
    for (int64_t k = nsteps - 1; k >= 0; --k, buf ^= 1) {
        const int64_t t0 = wk.t_begin + k * STEP;      // a block boundary
        const int64_t r0 = t0 + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;

        if constexpr (!PF) fetch_step(k, true, nxt);
        const StepIn in = nxt;
        if constexpr (PF) fetch_step(max(k - 1, (int64_t)0), k > 0, nxt);
        const R_* const xr = in.x;
        const R_* const br = in.b;
        const R_* const dyr = in.dy;
        const R_* const ar = in.a;
        float av[4][CPL], dh[4][CPL], az[4];
        if constexpr (PK > 1)
            decay_rows_packed<IO, CPL, kBwdDecay>(rsrc(ab + r0 * as), aoffp, (uint32_t)as, tr0, wk.t_begin, wk.t_end,
                                                  p.T, sig_a, az, av);
        else
            decay_rows<IO, CPL>(in.a, tr0, wk.t_begin, wk.t_end, p.T, sig_a, av);
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) dh[r][m] = dyr[r].get(m) * in.c[r].get(m);

        // ---- local solves: W = L (b*x), G; Dv = L^T (c*dy), Rr -------------------------
        float W[4][CPL], G[4][CPL], Dv[4][CPL], Rr[4][CPL];
        {
            float u[4][CPL];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int m = 0; m < CPL; ++m) u[r][m] = xr[r].get(m) * pregate(br[r].get(m), sig_b);
            chan_scan_fwd<CPL>(av, u, W, G, grp, lane);
        }
        chan_scan_rev<CPL>(av, dh, Dv, Rr, grp, lane);
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_wl[buf][wv][n * CPL + m] = W[3][m];
                s_cc[buf][wv][n * CPL + m] = G[3][m];
            }
        }
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_df[buf][wv][n * CPL + m] = av[0][m] * Dv[0][m];
        }
        if constexpr (VREC) prev_solve(t0, buf);
        lds_barrier();
        float vrec[CPL];   // kRecompute: the carrier of the block before the step
        if constexpr (VREC) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) vrec[m] = 0.f;
#pragma unroll 1
            for (int r = 0; r < TW; ++r) {   // the step before starts a block
                if ((r & smask) == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) vrec[m] = 0.f;
                }
                const int src = hw * TW + r;
#pragma unroll
                for (int m = 0; m < CPL; ++m)
                    vrec[m] = __builtin_fmaf(s_ccp[buf][src][n * CPL + m], vrec[m], s_wlp[buf][src][n * CPL + m]);
            }
        }
        const float* const vprev = VREC ? vrec : in.v;

        // ---- forward carriers entering this wave's sub-block ---------------------------
        float ein[CPL], sin_[CPL];
        {
            float e[CPL], s[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) { e[m] = SWR ? 0.f : vprev[m]; s[m] = SWR ? vprev[m] : 0.f; }
#pragma unroll 1
            for (int r = 0; r < tw; ++r) {
                if (SWR && (r & smask) == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                }
                const int src = hw * TW + r;
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float c_ = s_cc[buf][src][n * CPL + m];
                    const float wl = s_wl[buf][src][n * CPL + m];
                    e[m] = __builtin_fmaf(c_, e[m], wl);
                    if constexpr (SWR) s[m] = __builtin_fmaf(c_, s[m], wl);
                }
            }
            if (SWR && (tw & smask) == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
            }
#pragma unroll
            for (int m = 0; m < CPL; ++m) { ein[m] = e[m]; sin_[m] = s[m]; }
        }

        // ---- reverse carriers: capture at this sub-block, carry to the previous step ---
        float epsin[CPL], kd[CPL];
#pragma unroll 1
        for (int r = TW - 1; r >= 0; --r) {
            if (SWR && (r & smask) == smask) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            if (r == tw) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    epsin[m] = eps[m];
                    kd[m] = SWR ? (ein[m] - sin_[m]) * (eps[m] - pr[m]) : 0.f;
                }
            }
            const int src = hw * TW + r;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float c_ = s_cc[buf][src][n * CPL + m];
                const float df = s_df[buf][src][n * CPL + m];
                eps[m] = __builtin_fmaf(c_, eps[m], df);
                if constexpr (SWR) pr[m] = __builtin_fmaf(c_, pr[m], df);
            }
        }

        // ---- gradients -------------------------------------------------------------------
        float Gsh[4][CPL], hup[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            const float gprev = shfl(G[3][m], (lane - 16) & 63);   // G_{4grp-1}; G_{-1} = 1
            Gsh[0][m] = grp == 0 ? 1.0f : gprev;
#pragma unroll
            for (int r = 1; r < 4; ++r) Gsh[r][m] = G[r - 1][m];
#pragma unroll
            for (int r = 0; r < 4; ++r) W[r][m] = __builtin_fmaf(G[r][m], ein[m], W[r][m]);   // H: the jagged-window state
            const float hv = shfl(W[3][m], (lane - 16) & 63);
            hup[m] = grp == 0 ? ein[m] : hv;
        }
        const __amdgpu_buffer_rsrc_t rdx = rsrc(dxb + r0 * rs), rdb = rsrc(dbb + r0 * rs),
                                     rdc = rsrc(dcb + r0 * rs), rda = rsrc(dab + r0 * das);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float vdx[CPL], vdb[CPL], vdc[CPL], vda[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float dyv = dyr[r].get(m);
                vdc[m] = dyv * W[r][m];
                const float du = __builtin_fmaf(Rr[r][m], epsin[m], Dv[r][m]);
                const float zb = FEAT ? fresh(br[r].get(m)) : br[r].get(m);
                const SigSlope g = sig_b ? sigmoid_slope(zb) : SigSlope{zb, 1.0f};
                vdx[m] = g.s * du;
                if (p.residual) vdx[m] += dyv;
                vdb[m] = xr[r].get(m) * du * g.ds;
                vda[m] = __builtin_fmaf(r == 0 ? hup[m] : W[r - 1][m], du, -(Gsh[r][m] * Rr[r][m] * kd[m]));
                if (PK == 1 && sig_a) vda[m] *= sigmoid_slope(ar[r].get(m)).ds;
            }
            const uint32_t o = in_range(t < wk.t_end, loff + (uint32_t)(r * rs));
            store_row<IO, CPL, kBwdStore>(rdx, o, vdx);
            store_row<IO, CPL, kBwdStore>(rdb, o, vdb);
            store_row<IO, CPL, kBwdStore>(rdc, o, vdc);
            if constexpr (PK > 1) {
                // one decay per real head: sum over the head's channels (this
                // lane's and those of the head's other lanes of the row)
                float tot = 0.f;
#pragma unroll
                for (int m = 0; m < CPL; ++m) tot += vda[m];
#pragma unroll
                for (int w = 1; w < Geo<PK, CPL>::LPH; w <<= 1) tot += __shfl_xor(tot, w, 64);
                if (sig_a) tot *= sigmoid_slope(az[r]).ds;
                __builtin_amdgcn_raw_buffer_store_b32(
                    __builtin_bit_cast(int, tot), rda,
                    (int)in_range(t < wk.t_end && geo.lch == 0, daoff + (uint32_t)(r * das)), 0, kBwdStore);
            } else {
                store_row<IoF32, CPL, kBwdStore>(rda, in_range(t < wk.t_end, daoff + (uint32_t)(r * das)), vda);
            }
        }
    }
}

// Stage I of the exact backward with a per-channel decay: per run, the
// adjoint leaving its first token and the run's decay product, per channel.
template <class IO, int CPL, int TW, bool FEAT, int PK>
__global__ __launch_bounds__(TW * 64, 2) void swr_bwd_pc_agg_kernel(Params p) {
    const int sig_a = FEAT ? p.sig_a : 0;
    constexpr int D = CPL * SB;
    constexpr int STEP = TW * SB;
    constexpr int ES = IO::ES;
    using R_ = Row<IO, CPL>;
    __shared__ float s_df[2][TW][D];
    __shared__ float s_cc[2][TW][D];

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const Work wk = decode_work<1>(p, 0);
    const Geo<PK, CPL> geo(wk.h, p, n);
    const int64_t xo = (wk.b * p.sx_b + geo.head * p.sx_h + geo.coff) * ES;
    const char* cb = (const char*)p.c + xo;
    const char* dyb = (const char*)p.dy + xo;
    const char* ab = PK > 1 ? (const char*)p.a + (wk.b * p.sa_b + geo.head * p.sa_h) * ES : (const char*)p.a + xo;
    const int64_t rs = p.sx_t * ES;
    const int64_t as = PK > 1 ? p.sa_t * ES : rs;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoffp = (uint32_t)(4 * grp) * (uint32_t)as + (uint32_t)(geo.lh * p.sa_h * ES);
    const int64_t hb = wk.b * p.H + geo.head;

    float eps[CPL], prod[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { eps[m] = 0.f; prod[m] = 1.f; }
    int buf = 0;
    const int64_t nsteps = (wk.t_end - wk.t_begin + STEP - 1) / STEP;
    for (int64_t k = nsteps - 1; k >= 0; --k, buf ^= 1) {
        const int64_t r0 = wk.t_begin + k * STEP + tw * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs), ra = rsrc(ab + r0 * as);
        R_ cr[4], dyr[4], ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t o = in_range(tr0 + r < wk.t_end, loff + (uint32_t)(r * rs));
            cr[r].template load<kAggLoad>(rc, o);
            dyr[r].template load<kAggLoad>(rdy, o);
            if constexpr (PK == 1) ar[r].template load<kAggLoad>(ra, o);
        }
        float av[4][CPL], dh[4][CPL], Dv[4][CPL], R[4][CPL];
        if constexpr (PK > 1) {   // 1 past the end
            float az[4];
            decay_rows_packed<IO, CPL, kAggLoad>(ra, aoffp, (uint32_t)as, tr0, wk.t_begin, wk.t_end, p.T, sig_a, az, av);
        } else {
            decay_rows<IO, CPL>(ar, tr0, wk.t_begin, wk.t_end, p.T, sig_a, av);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int m = 0; m < CPL; ++m) dh[r][m] = dyr[r].get(m) * cr[r].get(m);
        chan_scan_rev<CPL>(av, dh, Dv, R, grp, lane);
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_df[buf][tw][n * CPL + m] = av[0][m] * Dv[0][m];
                s_cc[buf][tw][n * CPL + m] = av[0][m] * R[0][m];
            }
        }
        lds_barrier();
#pragma unroll 1
        for (int r = TW - 1; r >= 0; --r) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float c_ = s_cc[buf][r][n * CPL + m];
                prod[m] *= c_;
                eps[m] = c_ * eps[m] + s_df[buf][r][n * CPL + m];
            }
        }
    }
    const uint32_t o = in_range(tw == 0 && grp == 0, geo.off(p.nruns, wk.run) * 4u);
    store_row<IoF32, CPL>(rsrc(p.agg_v + hb * p.nruns * geo.Dr), o, eps);
    store_row<IoF32, CPL>(rsrc(p.agg_p + hb * p.nruns * geo.Dr), o, prod);
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

template <class IO, int CPL, bool FEAT, int MODE, int PK>
static hipError_t launch_pc(const Params& p, const Shape& sh, bool backward, hipStream_t stream) {
    const dim3 grid((unsigned)p.nwork);
#define SWR_LAUNCH(KERNEL, TW_, HW_)                                                                \
    else if (sh.tw == TW_ && sh.hw == HW_)                                                          \
        hipLaunchKernelGGL((KERNEL), grid, dim3(TW_ * HW_ * 64), 0, stream, p);
    if (backward) {
        if constexpr (MODE == kAggregate) {
            if (false) {}
            SWR_LAUNCH((swr_bwd_pc_agg_kernel<IO, CPL, 8, FEAT, PK>), 8, 1)
            SWR_LAUNCH((swr_bwd_pc_agg_kernel<IO, CPL, 4, FEAT, PK>), 4, 1)
            else return hipErrorInvalidValue;
        } else {
            if (false) {}
            SWR_LAUNCH((swr_bwd_pc_kernel<IO, CPL, 8, 1, FEAT, MODE, PK>), 8, 1)
            SWR_LAUNCH((swr_bwd_pc_kernel<IO, CPL, 4, 1, FEAT, MODE, PK>), 4, 1)
            else return hipErrorInvalidValue;
        }
    } else if constexpr (MODE != kRecompute) {   // (a backward-only mode)
        if (false) {}
        SWR_LAUNCH((swr_fwd_pc_kernel<IO, CPL, 4, 1, FEAT, MODE, PK>), 4, 1)
        SWR_LAUNCH((swr_fwd_pc_kernel<IO, CPL, 2, 2, FEAT, MODE, PK>), 2, 2)
        else return hipErrorInvalidValue;
    }
#undef SWR_LAUNCH
    return hipGetLastError();
}

template <class IO, int CPL, bool FEAT, int PK>
static hipError_t launch_pc_mode(const Params& p, const Shape& sh, bool backward, int mode, hipStream_t stream) {
    switch (mode) {
        case kSwr: return launch_pc<IO, CPL, FEAT, kSwr, PK>(p, sh, backward, stream);
        case kAggregate: return launch_pc<IO, CPL, FEAT, kAggregate, PK>(p, sh, backward, stream);
        case kExact: return launch_pc<IO, CPL, FEAT, kExact, PK>(p, sh, backward, stream);
        case kRecompute:
            if (!backward) return hipErrorInvalidValue;
            return launch_pc<IO, CPL, FEAT, kRecompute, PK>(p, sh, backward, stream);
        default: return hipErrorInvalidValue;
    }
}

template <class IO, int CPL, bool FEAT, int MODE>
static hipError_t launch_shape(const Params& p, const Shape& sh, bool backward, hipStream_t stream) {
    if constexpr (MODE == kPaired) {   // a forward-only mode
        if (backward) return hipErrorInvalidValue;
    }
    if constexpr (MODE == kRecompute) {
        if (!backward) return hipErrorInvalidValue;
    }
    const dim3 grid((unsigned)p.nwork);
#define SWR_LAUNCH(KERNEL, TW_, HW_)                                                                \
    else if (sh.tw == TW_ && sh.hw == HW_)                                                          \
        hipLaunchKernelGGL((KERNEL), grid, dim3(TW_ * HW_ * 64), 0, stream, p);
    if (backward) {
        if constexpr (MODE == kAggregate) {
            if (false) {}
            SWR_LAUNCH((swr_bwd_agg_kernel<IO, CPL, 8, FEAT>), 8, 1)
            SWR_LAUNCH((swr_bwd_agg_kernel<IO, CPL, 4, FEAT>), 4, 1)
            else return hipErrorInvalidValue;
        } else if constexpr (MODE != kPaired) {
            if (false) {}
            SWR_LAUNCH((swr_bwd_kernel<IO, CPL, 8, 1, FEAT, MODE>), 8, 1)
            SWR_LAUNCH((swr_bwd_kernel<IO, CPL, 4, 1, FEAT, MODE>), 4, 1)
            else return hipErrorInvalidValue;
        }
    } else if constexpr (MODE != kRecompute) {   // (a backward-only mode)
        if (false) {}
        SWR_LAUNCH((swr_fwd_kernel<IO, CPL, 4, 1, FEAT, MODE>), 4, 1)
        SWR_LAUNCH((swr_fwd_kernel<IO, CPL, 2, 2, FEAT, MODE>), 2, 2)
        else return hipErrorInvalidValue;
    }
#undef SWR_LAUNCH
    return hipGetLastError();
}

template <class IO, int CPL, bool FEAT>
static hipError_t launch_mode(const Params& p, const Shape& sh, bool backward, int mode, hipStream_t stream) {
    switch (mode) {
        case kSwr: return launch_shape<IO, CPL, FEAT, kSwr>(p, sh, backward, stream);
        case kAggregate: return launch_shape<IO, CPL, FEAT, kAggregate>(p, sh, backward, stream);
        case kExact: return launch_shape<IO, CPL, FEAT, kExact>(p, sh, backward, stream);
        case kGrouped: return launch_shape<IO, CPL, FEAT, kGrouped>(p, sh, backward, stream);
        case kRecompute: return launch_shape<IO, CPL, FEAT, kRecompute>(p, sh, backward, stream);
        case kPaired:
            if constexpr (CPL == 8 && IO::ES == 2) return launch_shape<IO, CPL, FEAT, kPaired>(p, sh, backward, stream);
            return hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

template <class IO, bool FEAT>
static hipError_t launch_cpl(const Params& p, int D, const Shape& sh, bool backward, bool per_channel,
                             int pack, int mode, hipStream_t stream) {
    if (pack > 1) {   // packed small heads: 64-channel virtual heads of 4 or 2 real heads
        if (D != 64) return hipErrorInvalidValue;
        return pack == 4 ? launch_pc_mode<IO, 4, FEAT, 4>(p, sh, backward, mode, stream)
                         : launch_pc_mode<IO, 4, FEAT, 2>(p, sh, backward, mode, stream);
    }
    if (per_channel) {
        switch (D) {   // channels of a virtual head (at most 64)
            case 16: return launch_pc_mode<IO, 1, FEAT, 1>(p, sh, backward, mode, stream);
            case 32: return launch_pc_mode<IO, 2, FEAT, 1>(p, sh, backward, mode, stream);
            case 64: return launch_pc_mode<IO, 4, FEAT, 1>(p, sh, backward, mode, stream);
            default: return hipErrorInvalidValue;
        }
    }
    switch (D) {
        case 16: return launch_mode<IO, 1, FEAT>(p, sh, backward, mode, stream);
        case 32: return launch_mode<IO, 2, FEAT>(p, sh, backward, mode, stream);
        case 64: return launch_mode<IO, 4, FEAT>(p, sh, backward, mode, stream);
        case 128: return launch_mode<IO, 8, FEAT>(p, sh, backward, mode, stream);
        default: return hipErrorInvalidValue;
    }
}

// Kernels without the featurisation code are separate instantiations, so the
// plain path carries none of its registers.
template <class IO>
static hipError_t launch_feat(const Params& p, int D, const Shape& sh, bool backward, bool per_channel,
                              int pack, int mode, hipStream_t stream) {
    if (p.sig_a || p.sig_b) return launch_cpl<IO, true>(p, D, sh, backward, per_channel, pack, mode, stream);
    return launch_cpl<IO, false>(p, D, sh, backward, per_channel, pack, mode, stream);
}

// Zeroes da ([B, T, H] float32 with a's strides) before the virtual heads of
// a split head add their shares of the decay gradient.
__global__ __launch_bounds__(256) void swr_da_zero_kernel(float* da, int64_t T, int64_t H, int64_t sa_b,
                                                          int64_t sa_t, int64_t sa_h, int64_t total) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t h = i % H, t = (i / H) % T, b = i / (H * T);
        da[b * sa_b + t * sa_t + h * sa_h] = 0.0f;
    }
}

hipError_t launch(const Params& p, int dtype, int D, const Shape& sh, bool backward, bool per_channel,
                  int pack, int mode, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    if (backward && !per_channel && pack == 1 && p.hshift > 0) {
        if (mode != kSwr && mode != kRecompute) return hipErrorInvalidValue;
        const int64_t total = p.B * p.T * p.H;
        const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
        hipLaunchKernelGGL(swr_da_zero_kernel, dim3((uint32_t)blocks), dim3(256), 0, st, p.da, p.T, p.H, p.sa_b,
                           p.sa_t, p.sa_h, total);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dtype == 1) return launch_feat<IoBf16>(p, D, sh, backward, per_channel, pack, mode, st);
    return launch_feat<IoF32>(p, D, sh, backward, per_channel, pack, mode, st);
}

template <class IO, int CPL>
static hipError_t launch_step_cpl(const StepParams& q, bool exact, bool pc, bool feat, hipStream_t st) {
    const int64_t n = q.B * q.H * 16;
    const dim3 grid((unsigned)((n + 255) / 256)), blk(256);
    const int sel = (exact ? 4 : 0) | (pc ? 2 : 0) | (feat ? 1 : 0);
    switch (sel) {
        case 0: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, false, false, false>), grid, blk, 0, st, q); break;
        case 1: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, false, false, true>), grid, blk, 0, st, q); break;
        case 2: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, false, true, false>), grid, blk, 0, st, q); break;
        case 3: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, false, true, true>), grid, blk, 0, st, q); break;
        case 4: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, true, false, false>), grid, blk, 0, st, q); break;
        case 5: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, true, false, true>), grid, blk, 0, st, q); break;
        case 6: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, true, true, false>), grid, blk, 0, st, q); break;
        default: hipLaunchKernelGGL((swr_step_kernel<IO, CPL, true, true, true>), grid, blk, 0, st, q); break;
    }
    return hipGetLastError();
}

template <class IO>
static hipError_t launch_step_io(const StepParams& q, int D, bool exact, bool pc, hipStream_t st) {
    const bool feat = q.sig_a || q.sig_b;
    switch (D) {
        case 16: return launch_step_cpl<IO, 1>(q, exact, pc, feat, st);
        case 32: return launch_step_cpl<IO, 2>(q, exact, pc, feat, st);
        case 64: return launch_step_cpl<IO, 4>(q, exact, pc, feat, st);
        case 128: return launch_step_cpl<IO, 8>(q, exact, pc, feat, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_step(const StepParams& q, int dtype, int D, bool exact, bool per_channel, void* stream) {
    if (q.B * q.H == 0) return hipSuccess;
    hipStream_t st = (hipStream_t)stream;
    if (dtype == 1) return launch_step_io<IoBf16>(q, D, exact, per_channel, st);
    return launch_step_io<IoF32>(q, D, exact, per_channel, st);
}

template <class IO, int CPL>
static hipError_t launch_state_cpl(const StateParams& q, bool pc, hipStream_t st) {
    const int64_t n = q.B * q.H * 16;
    const dim3 grid((unsigned)((n + 255) / 256)), blk(256);
    const int sel = (pc ? 2 : 0) | (q.sig_a ? 1 : 0);
    switch (sel) {
        case 0: hipLaunchKernelGGL((swr_state_kernel<IO, CPL, false, false>), grid, blk, 0, st, q); break;
        case 1: hipLaunchKernelGGL((swr_state_kernel<IO, CPL, false, true>), grid, blk, 0, st, q); break;
        case 2: hipLaunchKernelGGL((swr_state_kernel<IO, CPL, true, false>), grid, blk, 0, st, q); break;
        default: hipLaunchKernelGGL((swr_state_kernel<IO, CPL, true, true>), grid, blk, 0, st, q); break;
    }
    return hipGetLastError();
}

template <class IO>
static hipError_t launch_state_io(const StateParams& q, int D, bool pc, hipStream_t st) {
    switch (D) {
        case 16: return launch_state_cpl<IO, 1>(q, pc, st);
        case 32: return launch_state_cpl<IO, 2>(q, pc, st);
        case 64: return launch_state_cpl<IO, 4>(q, pc, st);
        case 128: return launch_state_cpl<IO, 8>(q, pc, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_state(const StateParams& q, int dtype, int D, bool per_channel, void* stream) {
    if (q.B * q.H == 0) return hipSuccess;
    hipStream_t st = (hipStream_t)stream;
    if (dtype == 1) return launch_state_io<IoBf16>(q, D, per_channel, st);
    return launch_state_io<IoF32>(q, D, per_channel, st);
}

template <class IO>
static hipError_t launch_gate_reduce_io(const Params& p, int D, hipStream_t st) {
    const int64_t n = p.B * p.T * (p.H / p.group) * 16;
    const dim3 grid((unsigned)((n + 255) / 256)), blk(256);
    switch (D) {
        case 16: hipLaunchKernelGGL((swr_gate_reduce_kernel<IO, 1>), grid, blk, 0, st, p); break;
        case 32: hipLaunchKernelGGL((swr_gate_reduce_kernel<IO, 2>), grid, blk, 0, st, p); break;
        case 64: hipLaunchKernelGGL((swr_gate_reduce_kernel<IO, 4>), grid, blk, 0, st, p); break;
        case 128: hipLaunchKernelGGL((swr_gate_reduce_kernel<IO, 8>), grid, blk, 0, st, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gate_reduce(const Params& p, int dtype, int D, void* stream) {
    if (p.B * p.T * p.H == 0) return hipSuccess;
    hipStream_t st = (hipStream_t)stream;
    return dtype == 1 ? launch_gate_reduce_io<IoBf16>(p, D, st) : launch_gate_reduce_io<IoF32>(p, D, st);
}

hipError_t launch_scan(const ScanParams& q, void* stream) {
    const int64_t n = q.seqs * q.D;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(swr_scan_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream, q);
    return hipGetLastError();
}

}  // namespace swr
