// swr_chain.hip -- the exact (untruncated) recurrence in one pass: the
// forward (a decay per head or per channel), and the backward for heads of
// up to 64 channels.
//
// The three-stage evaluation of the hierarchical decomposition (Alg.
// "Hierarchical Block Parallel Inference": local solves, the carrier
// recurrence, reconstruction) reads x, b and a twice.  Here the carrier
// recurrence is resolved while the chunks are processed, by a look-back
// between workgroups: each chunk of 128 tokens of a sequence is solved locally
// from zero, which gives its aggregate, the end state V and decay product P of
// the chunk started from zero.  The state entering chunk c is then
//   S_c = P_{c-1} ( ... P_{k+1} (P_k S_k' + V_k) ...) + V_{c-1},
// composed from the inclusive end state S_k' of the last boundary chunk k
// before c (every 16th chunk, or every 8th; before the first one, the
// initial state) and the aggregates of the chunks in between.  Boundary chunks publish their
// inclusive end state P S + V, the others their aggregate.  The composition
// always takes the same chunks in the same pattern, so the results do not
// depend on the order in which workgroups reach them; the outputs then follow
// from the chunk's local solves, kept in registers or LDS.  Every input is
// read once (x twice with the residual and bf16 heads of 64 or 128).
//
// Chunks are handed out in order by a ticket counter (chunk-major over the
// sequences), so a chunk only ever waits for chunks of lower tickets, whose
// workgroups are already running.  A wait is bounded: past p.spin_limit polls
// (2^16 unless the host lowers it) the chunk counts the time-out and proceeds
// from a NaN state, so that a lost publication (never expected) shows in
// every output that depends on it instead of passing as a plausible value.
//
// Publication uses device-coherent (agent-scope) stores, and a wait for
// their completion before the flag that announces them; readers load the flag
// and then the data with device-coherent loads.  The backward runs the same
// chain from each sequence's end, on the adjoint entering a chunk from its
// end.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swr_device.h"
#include "swr_launch.h"

namespace swr {
namespace {

constexpr int kChainTW = 8;                // waves per workgroup, one sub-block each
constexpr int kChainTok = kChainTW * SB;   // tokens per chunk
constexpr int kFlagAgg = 1, kFlagIncl = 2;
// Chunks K - 1, 2 K - 1, ... of a sequence publish their inclusive end state,
// the others their aggregate; every chunk composes the aggregates since the
// last such boundary, Q per lane group (four groups, K = 4 Q), loaded QB at a
// time: 2 where the kernel is held to 80 registers, else 4.  A longer K
// shortens the chain of boundaries; a second batch of loads lengthens every
// chunk's look-back: Q = 2 (one batch) for the 80-register kernels on
// sequences shorter than kLongChain chunks, else Q = 4.
constexpr int64_t kLongChain = 256;
template <int CPL, bool WL>
constexpr int chain_qb() { return WL && CPL <= 4 ? 2 : 4; }
// device-coherent (sc1) vector loads of published values
constexpr int kCoherent = 16;

__device__ inline void put_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void put_flag(int32_t* p, int v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline int get_flag(const int32_t* p) {
    return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until this wave's memory writes are complete (vmcnt(0)); the
// compiler moves no memory access across it.
__device__ inline void writes_complete() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// bf16 lanes of 8 or 16 channels (heads of 64 and 128): the local solutions
// wait for the look-back in LDS instead of registers, and x is loaded again
// for the residual, so that the kernel fits 128 registers (two workgroups a
// compute unit) or 80 (three); the launcher sizes its grid to match.
template <class IO, int CPL>
constexpr bool chain_w_in_lds() { return (CPL == 8 || CPL == 4) && IO::ES == 2; }
template <class IO, int CPL>
constexpr int chain_waves_per_simd() { return chain_w_in_lds<IO, CPL>() ? (CPL == 8 ? 4 : 6) : 1; }

// How a chunk's decay product is kept: one value a chunk (a decay per head),
// one per lane column (heads taken two at a time: lanes n < 8 and n >= 8
// belong to different heads), or one per channel (a decay per channel).
enum ChainP { kPChunk, kPLane, kPChannel };

// Wave 0's part in the chain for chunk ci of a sequence (chunks slot0 ...
// slot0 + nch - 1 of the workspace arrays, in chain order): publish the
// chunk's aggregate (V, P), wait for the last boundary's inclusive value and
// the aggregates after it, compose them in a fixed pattern (lane group g
// folds chunks kb+1+Q*g ... kb+Q*(g+1) in order, then the groups' results
// are applied to the boundary value in order), and at a boundary publish the
// chunk's own inclusive value.  `in` is the value entering the chain's first
// chunk (this lane's slice at in + n * CPL; NULL for zero).  Returns the
// value entering the chunk and the one leaving it (I = P in + V).  P holds
// CPL values with kPChannel, else one.
template <int CPL, int Q, int QB, int PM>
__device__ inline void chain_link(const Params& p, int64_t slot0, int64_t ci, int64_t nch, const float (&V)[CPL],
                                  const float (&P)[PM == kPChannel ? CPL : 1], const float* in, int lane, int grp,
                                  int n, float (&pre)[CPL], float (&I)[CPL]) {
    constexpr int D = CPL * SB, K = 4 * Q;
    constexpr int NP = PM == kPChannel ? CPL : 1;                      // values a lane keeps
    constexpr int PD = PM == kPChannel ? D : PM == kPLane ? SB : 1;    // values a chunk stores
    const uint32_t vch = (uint32_t)(n * CPL);
    const uint32_t pch = PM == kPChannel ? vch : PM == kPLane ? (uint32_t)n : 0u;   // this lane's first
    const int64_t slot = slot0 + ci;
    const bool boundary = ci % K == K - 1;
    // the last boundary chunk before this one (or none), and the chunks in between
    const int64_t kb = ci / K * K - 1;
    const int cnt = (int)(ci - 1 - kb);
    if (!boundary && ci + 1 < nch) {   // later chunks of the group compose this aggregate
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) put_coherent(p.agg_v + slot * D + vch + m, V[m]);
            if constexpr (PM != kPChunk) {
#pragma unroll
                for (int m = 0; m < NP; ++m) put_coherent(p.agg_p + slot * PD + pch + m, P[m]);
            }
        }
        if (PM == kPChunk && lane == 0) put_coherent(p.agg_p + slot, P[0]);
        writes_complete();
        if (lane == 0) put_flag(p.chain_flags + slot, kFlagAgg);
    }
    // wait until the boundary's inclusive value and the aggregates in
    // between are published: lane i < cnt polls chunk kb + 1 + i, lane 63 the boundary
    bool timed_out = false;
    int spins = 0;
#pragma unroll 1
    for (;;) {
        bool ok = true;
        if (lane < cnt)
            ok = get_flag(p.chain_flags + slot0 + kb + 1 + lane) == kFlagAgg;
        else if (lane == 63 && kb >= 0)
            ok = get_flag(p.chain_flags + slot0 + kb) == kFlagIncl;
        if (__all(ok)) break;
        if (++spins > p.spin_limit) {   // never expected: count it, poison the outputs
            if (lane == 0) atomicAdd(p.chain_ctr + 1, 1);
            timed_out = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    float gV[CPL], gP[NP];
#pragma unroll
    for (int m = 0; m < CPL; ++m) gV[m] = 0.f;
#pragma unroll
    for (int m = 0; m < NP; ++m) gP[m] = 1.0f;
    {
        const __amdgpu_buffer_rsrc_t rav = rsrc(p.agg_v + slot0 * D), rap = rsrc(p.agg_p + slot0 * PD);
#pragma unroll
        for (int q0 = 0; q0 < Q; q0 += QB) {   // QB aggregates in flight at a time
            Row<IoF32, CPL> rv[QB];
            Row<IoF32, NP> rp[QB];
#pragma unroll
            for (int q = 0; q < QB; ++q) {
                const int i = grp * Q + q0 + q;
                const int64_t j = kb + 1 + i;
                rv[q].template load<kCoherent>(rav, in_range(i < cnt, (uint32_t)(j * D + vch) * 4u));
                rp[q].template load<kCoherent>(rap, in_range(i < cnt, (uint32_t)(j * PD + pch) * 4u));
            }
#pragma unroll
            for (int q = 0; q < QB; ++q) {
                const bool live = grp * Q + q0 + q < cnt;
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float pq = live ? rp[q].get(NP > 1 ? m : 0) : 1.0f;
                    gV[m] = __builtin_fmaf(pq, gV[m], rv[q].get(m));
                }
#pragma unroll
                for (int m = 0; m < NP; ++m) gP[m] *= live ? rp[q].get(m) : 1.0f;
            }
            if constexpr (QB < Q) __builtin_amdgcn_sched_barrier(0);   // one batch live at a time
        }
    }
    // the boundary's inclusive value, or the chain's entering value (zero without one)
    {
        Row<IoF32, CPL> ri;
        if (kb >= 0)
            ri.template load<kCoherent>(rsrc(p.chain_incl + slot0 * D), (uint32_t)(kb * D + vch) * 4u);
        else
            ri.load(rsrc(in ? in : p.chain_incl), in_range(in != nullptr, vch * 4u));
#pragma unroll
        for (int m = 0; m < CPL; ++m) pre[m] = ri.get(m);
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int src = g * 16 + n;
        float pg[NP];
#pragma unroll
        for (int m = 0; m < NP; ++m) pg[m] = __shfl(gP[m], src);
#pragma unroll
        for (int m = 0; m < CPL; ++m) pre[m] = __builtin_fmaf(pg[NP > 1 ? m : 0], pre[m], __shfl(gV[m], src));
    }
    if (timed_out) {
#pragma unroll
        for (int m = 0; m < CPL; ++m) pre[m] = __builtin_nanf("");
    }
#pragma unroll
    for (int m = 0; m < CPL; ++m) I[m] = __builtin_fmaf(P[NP > 1 ? m : 0], pre[m], V[m]);
    if (boundary && ci + 1 < nch) {
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) put_coherent(p.chain_incl + slot * D + vch + m, I[m]);
        }
        writes_complete();
        if (lane == 0) put_flag(p.chain_flags + slot, kFlagIncl);
    }
}

template <class IO, int CPL, bool FEAT, int Q>
__global__ __launch_bounds__(kChainTW * 64, (chain_waves_per_simd<IO, CPL>())) void swr_fwd_chain_kernel(Params p) {
    constexpr int TW = kChainTW;
    constexpr int TOK = kChainTok;
    constexpr int D = CPL * SB;
    constexpr int ES = IO::ES;
    using RW = Row<IO, CPL>;
    constexpr bool WL = chain_w_in_lds<IO, CPL>();
    constexpr int QB = chain_qb<CPL, WL>();
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;
    __shared__ float s_wl[TW][D];   // last row of each sub-block's local solve
    __shared__ float s_c[TW];       // decay product of each sub-block
    __shared__ float s_pre[D];      // the exact state entering the chunk
    __shared__ f32x4 s_W[WL ? TW : 1][WL ? CPL : 1][WL ? 64 : 1];   // WL: each lane's local solution
    __shared__ int64_t s_ticket[2];

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    // (virtual) sequences: a head of p.dh channels is 2^hshift virtual heads of D
    const int64_t S = p.B * p.Hv, nch = p.nruns, N = S * nch;
    const int hmask = (1 << p.hshift) - 1;
    const int64_t DH = p.dh;
    const int64_t rs = p.sx_t * ES, as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const int smask = p.block / SB - 1;

    // Tickets pass through LDS; two slots, so that a slot is only rewritten
    // after a later barrier has ordered every wave's read of it.
    int par = 0;
    auto grab = [&]() {
        if (threadIdx.x == 0) s_ticket[par] = atomicAdd(p.chain_ctr, 1);
        lds_barrier();
        const int64_t t = s_ticket[par];
        par ^= 1;
        return t;
    };
    int64_t ticket = grab();
    for (;;) {
        if (ticket >= N) break;
        const int64_t seq = ticket % S, ch = ticket / S;   // chunk-major: earlier chunks first
        const int64_t slot = seq * nch + ch;
        const int64_t rseq = seq >> p.hshift;   // the real (batch, head) sequence
        const int64_t coff = (int64_t)(seq & hmask) * D;   // its first channel here
        const int64_t xo = (rseq / p.H * p.sx_b + rseq % p.H * p.sx_h + coff) * ES;
        const int64_t t0 = ch * TOK, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;

        // ---- the sub-block's local solve W = L u ----------------------------------
        RW xr[4], br[4], cr[4];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs),
                                         rb = rsrc((const char*)p.b + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs));
                xr[r].template load<kFwdLoad>(rx, o);
                br[r].template load<kFwdLoad>(rb, o);
            }
        }
        const bool a_ok = r0 + n < p.T;
        float a_n = load_scalar<IO, kFwdDecay>(
            rsrc((const char*)p.a + (rseq / p.H * p.sa_b + rseq % p.H * p.sa_h) * ES + r0 * as), in_range(a_ok, aoff));
        if (sig_a) a_n = sigmoid(a_n);
        if (!a_ok) a_n = 1.0f;   // past the sequence's end the state is carried unchanged
        const Decay dk = build_decay(a_n, grp, n);
        f32x4 W[CPL];
        {
            const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
                W[m] = Contract<IO>::run(A, u);
            }
        }
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[tw][n * CPL + m] = W[m][3];
        }
        if (lane == 63) s_c[tw] = dk.c;
        if constexpr (WL) {   // (read back by the same lane)
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_W[tw][m][lane] = W[m];
        }
        {   // c is needed for the outputs only: its loads go out now and land during the look-back
            const __amdgpu_buffer_rsrc_t rc = rsrc((const char*)p.c + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                cr[r].template load<kFwdLoad>(rc, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)));
        }
        lds_barrier();

        // ---- wave 0: the chunk's aggregate, the look-back, the inclusive state -----
        if (tw == 0) {
            float V[CPL], P = 1.0f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) V[m] = 0.f;
#pragma unroll 1
            for (int r = 0; r < TW; ++r) {
                const float c_ = s_c[r];
#pragma unroll
                for (int m = 0; m < CPL; ++m) V[m] = __builtin_fmaf(c_, V[m], s_wl[r][n * CPL + m]);
                P *= c_;
            }
            const uint32_t vch = (uint32_t)(n * CPL);
            float pre[CPL], I[CPL];
            const float Pv[1] = {P};
            chain_link<CPL, Q, QB, kPChunk>(p, seq * nch, ch, nch, V, Pv, p.h0 ? p.h0 + rseq * DH + coff : nullptr,
                                          lane, grp, n, pre, I);
            if (grp == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_pre[vch + m] = pre[m];
            }
            store_row<IoF32, CPL>(rsrc(p.h_last ? p.h_last + rseq * DH + coff : p.chain_incl),
                                  in_range(p.h_last && ch == nch - 1 && grp == 0, (uint32_t)vch * 4u), I);
        }
        lds_barrier();

        // ---- outputs: the state entering this wave's sub-block, y, block carriers -----
        float e[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) e[m] = s_pre[n * CPL + m];
#pragma unroll 1
        for (int r = 0; r < tw; ++r) {
            const float c_ = s_c[r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) e[m] = __builtin_fmaf(c_, e[m], s_wl[r][n * CPL + m]);
        }
        const __amdgpu_buffer_rsrc_t ry = rsrc((char*)p.y + xo + r0 * rs);
        f32x4 Wo[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            if constexpr (WL) Wo[m] = s_W[tw][m][lane];
            else Wo[m] = W[m];
        }
        RW xres[4];   // the residual's x: WL loads it again rather than keep it through the look-back
        if constexpr (WL) {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                xres[r].template load<kFwdLoad>(rx, in_range(p.residual && tr0 + r < p.T, loff + (uint32_t)(r * rs)));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) xres[r] = xr[r];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                yv[m] = cr[r].get(m) * __builtin_fmaf(dk.G[r], e[m], Wo[m][r]);
                if (p.residual) yv[m] += xres[r].get(m);
            }
            store_row<IO, CPL, kFwdStore>(ry, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)), yv);
        }
        // the exact state at the end of a block that ends with this sub-block
        // (a block longer than a chunk that the sequence's end cuts short ends in the last chunk)
        if (p.carriers && (((ch * TW + tw) & smask) == smask || (ch == nch - 1 && tw == TW - 1))) {
            const int64_t blk = r0 >> p.lshift;
            float v[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) v[m] = __builtin_fmaf(dk.c, e[m], s_wl[tw][n * CPL + m]);
            store_row<IoF32, CPL>(rsrc(p.carriers + (rseq * p.nblocks * DH + coff)),
                                  in_range(grp == 0 && blk < p.nblocks, (uint32_t)(blk * DH + n * CPL) * 4u), v);
        }
        ticket = grab();
    }
}

// The exact forward in one pass for bf16 heads of 64 channels taken two at a
// time (adjacent heads h, h+1 of an even head count): lanes n < 8 hold
// head h's channels and n >= 8 head h+1's, so that every lane moves a
// 16-byte row slice, as in the jagged window's paired forward.  Each head
// has its own decay operator (two MFMA solves, each lane keeping its head's
// result) and decay products; the chain runs over the pair with a decay
// product per channel.  The local solutions wait for the look-back in LDS
// (two workgroups a compute unit).
template <bool FEAT, int Q>
__global__ __launch_bounds__(kChainTW * 64, 4) void swr_fwd_chain_pair_kernel(Params p) {
    using IO = IoBf16;
    constexpr int CPL = 8;
    constexpr int TW = kChainTW;
    constexpr int TOK = kChainTok;
    constexpr int D = CPL * SB;   // the pair's 128 channels
    constexpr int DH = D / 2;     // channels of one head
    constexpr int ES = IO::ES;
    using RW = Row<IO, CPL>;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;
    __shared__ float s_wl[TW][D];   // last row of each sub-block's local solve
    __shared__ float s_c[TW][2];    // decay product of each sub-block, per head
    __shared__ float s_pre[D];      // the exact state entering the chunk
    __shared__ f32x4 s_W[TW][CPL][64];
    __shared__ int64_t s_ticket[2];

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const int hsel = n >> 3;   // this lane's head of the pair
    const int64_t HP = p.H / 2, S = p.B * HP, nch = p.nruns, N = S * nch;
    const int64_t rs = p.sx_t * ES, as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(hsel * p.sx_h * ES) +
                          (uint32_t)((n & 7) * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const uint32_t vch = (uint32_t)(n * CPL);   // this lane's slice of the pair's [2][64] states
    const int smask = p.block / SB - 1;

    int par = 0;
    auto grab = [&]() {
        if (threadIdx.x == 0) s_ticket[par] = atomicAdd(p.chain_ctr, 1);
        lds_barrier();
        const int64_t t = s_ticket[par];
        par ^= 1;
        return t;
    };
    int64_t ticket = grab();
    for (;;) {
        if (ticket >= N) break;
        const int64_t seq = ticket % S, ch = ticket / S;   // chunk-major: earlier chunks first
        const int64_t bi = seq / HP, h0 = 2 * (seq % HP);  // the pair's first head
        const int64_t xo = (bi * p.sx_b + h0 * p.sx_h) * ES;
        const int64_t t0 = ch * TOK, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;

        // ---- the sub-block's local solves, one operator per head ----------------------
        RW xr[4], br[4], cr[4];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs),
                                         rb = rsrc((const char*)p.b + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs));
                xr[r].template load<kFwdLoad>(rx, o);
                br[r].template load<kFwdLoad>(rb, o);
            }
        }
        const bool a_ok = r0 + n < p.T;
        const char* ab = (const char*)p.a + (bi * p.sa_b + h0 * p.sa_h) * ES + r0 * as;
        float a_n = load_scalar<IO, kFwdDecay>(rsrc(ab), in_range(a_ok, aoff));
        float a_n1 = load_scalar<IO, kFwdDecay>(rsrc(ab + p.sa_h * ES), in_range(a_ok, aoff));
        if (sig_a) { a_n = sigmoid(a_n); a_n1 = sigmoid(a_n1); }
        if (!a_ok) { a_n = 1.0f; a_n1 = 1.0f; }   // past the sequence's end the state is carried unchanged
        const Decay dk = build_decay(a_n, grp, n), dk1 = build_decay(a_n1, grp, n);
        float Gl[4];   // this lane's head's prefix products at its rows
#pragma unroll
        for (int r = 0; r < 4; ++r) Gl[r] = hsel ? dk1.G[r] : dk.G[r];
        const float cl = hsel ? dk1.c : dk.c;
        {
            const typename Contract<IO>::A A = Contract<IO>::prep(dk.L), A1 = Contract<IO>::prep(dk1.L);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * pregate(br[q].get(m), sig_b);
                const f32x4 W0 = Contract<IO>::run(A, u), W1 = Contract<IO>::run(A1, u);
                const f32x4 W = hsel ? W1 : W0;   // each lane keeps its own head's result
                if (grp == 3) s_wl[tw][vch + m] = W[3];
                s_W[tw][m][lane] = W;             // (read back by the same lane)
            }
        }
        if (lane == 63) { s_c[tw][0] = dk.c; s_c[tw][1] = dk1.c; }
        {   // c is needed for the outputs only: its loads land during the look-back
            const __amdgpu_buffer_rsrc_t rc = rsrc((const char*)p.c + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                cr[r].template load<kFwdLoad>(rc, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)));
        }
        lds_barrier();

        // ---- wave 0: the chunk's aggregate, the look-back, the inclusive state -----
        if (tw == 0) {
            float V[CPL], P = 1.0f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) V[m] = 0.f;
#pragma unroll 1
            for (int r = 0; r < TW; ++r) {
                const float c_ = s_c[r][hsel];
#pragma unroll
                for (int m = 0; m < CPL; ++m) V[m] = __builtin_fmaf(c_, V[m], s_wl[r][vch + m]);
                P *= c_;
            }
            const float Pv[1] = {P};
            float pre[CPL], I[CPL];
            const int64_t so = (bi * p.H + h0) * DH;   // the pair's two [64] state rows, adjacent
            chain_link<CPL, Q, 2, kPLane>(p, seq * nch, ch, nch, V, Pv, p.h0 ? p.h0 + so : nullptr, lane, grp, n,
                                          pre, I);
            if (grp == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_pre[vch + m] = pre[m];
            }
            store_row<IoF32, CPL>(rsrc(p.h_last ? p.h_last + so : p.chain_incl),
                                  in_range(p.h_last && ch == nch - 1 && grp == 0, vch * 4u), I);
        }
        lds_barrier();

        // ---- outputs: the state entering this wave's sub-block, y, block carriers -----
        float e[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) e[m] = s_pre[vch + m];
#pragma unroll 1
        for (int r = 0; r < tw; ++r) {
            const float c_ = s_c[r][hsel];
#pragma unroll
            for (int m = 0; m < CPL; ++m) e[m] = __builtin_fmaf(c_, e[m], s_wl[r][vch + m]);
        }
        const __amdgpu_buffer_rsrc_t ry = rsrc((char*)p.y + xo + r0 * rs);
        RW xres[4];   // the residual's x, loaded again rather than kept through the look-back
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                xres[r].template load<kFwdLoad>(rx, in_range(p.residual && tr0 + r < p.T, loff + (uint32_t)(r * rs)));
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const f32x4 W = s_W[tw][m][lane];
                yv[m] = cr[r].get(m) * __builtin_fmaf(Gl[r], e[m], W[r]);
                if (p.residual) yv[m] += xres[r].get(m);
            }
            store_row<IO, CPL, kFwdStore>(ry, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)), yv);
        }
        // the exact state at the end of a block that ends with this sub-block
        // (a block longer than a chunk that the sequence's end cuts short ends in the last chunk)
        if (p.carriers && (((ch * TW + tw) & smask) == smask || (ch == nch - 1 && tw == TW - 1))) {
            const int64_t blk = r0 >> p.lshift;
            float v[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) v[m] = __builtin_fmaf(cl, e[m], s_wl[tw][vch + m]);
            // each head's rows [nblocks][64]; this lane's head's, then its block's, slice
            store_row<IoF32, CPL>(rsrc(p.carriers + (bi * p.H + h0) * p.nblocks * DH),
                                  in_range(grp == 0 && blk < p.nblocks,
                                           (uint32_t)((hsel * p.nblocks + blk) * DH + (n & 7) * CPL) * 4u), v);
        }
        ticket = grab();
    }
}

// The exact forward in one pass with a decay per channel (heads of 128 as
// two virtual heads of 64).  The chunks' local solves are the per-lane scans
// of the per-channel sweep kernels (whose lane geometry, Geo, also covers
// packed small heads: PK heads of 64 / PK channels a virtual head); the chain
// is that of swr_fwd_chain_kernel with the decay products kept per channel.
// (Lanes of 4 channels park their local solution and prefix products in LDS
// through the look-back, 64 KB a workgroup, so that two workgroups share a
// compute unit.)
template <class IO, int CPL, bool FEAT, int PK, int Q>
__global__ __launch_bounds__(kChainTW * 64, (CPL == 4 ? 4 : 2)) void swr_fwd_chain_pc_kernel(Params p) {
    constexpr int TW = kChainTW;
    constexpr int TOK = kChainTok;
    constexpr int D = CPL * SB;
    constexpr int ES = IO::ES;
    constexpr bool PARK = CPL == 4;
    using RW = Row<IO, CPL>;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;
    __shared__ float s_wl[TW][D];   // last row of each sub-block's local solve
    __shared__ float s_cc[TW][D];   // each sub-block's decay product, per channel
    __shared__ float s_pre[D];      // the exact state entering the chunk
    __shared__ f32x4 s_WG[PARK ? TW : 1][PARK ? 2 * CPL : 1][PARK ? 64 : 1];
    __shared__ int64_t s_ticket[2];

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const int64_t S = p.B * p.Hv, nch = p.nruns, N = S * nch;
    const int64_t rs = p.sx_t * ES, as = PK > 1 ? p.sa_t * ES : rs;
    const uint32_t vch = (uint32_t)(n * CPL);
    const int smask = p.block / SB - 1;

    int par = 0;
    auto grab = [&]() {
        if (threadIdx.x == 0) s_ticket[par] = atomicAdd(p.chain_ctr, 1);
        lds_barrier();
        const int64_t t = s_ticket[par];
        par ^= 1;
        return t;
    };
    int64_t ticket = grab();
    for (;;) {
        if (ticket >= N) break;
        const int64_t seq = ticket % S, ch = ticket / S;   // chunk-major: earlier chunks first
        const int64_t bi = seq / p.Hv, vh = seq % p.Hv;
        const Geo<PK, CPL> geo(vh, p, n);
        const int64_t hb = bi * p.H + geo.head;   // first real (batch, head) of the virtual head
        const int64_t xo = (bi * p.sx_b + geo.head * p.sx_h + geo.coff) * ES;
        const char* ab = PK > 1 ? (const char*)p.a + (bi * p.sa_b + geo.head * p.sa_h) * ES : (const char*)p.a + xo;
        const uint32_t loff = in_range(geo.ok, (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES));
        const uint32_t aoffp = (uint32_t)(4 * grp) * (uint32_t)as + (uint32_t)(geo.lh * p.sa_h * ES);
        const int64_t t0 = ch * TOK, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;

        // ---- the sub-block's local solve: per-lane scans ------------------------------
        RW xr[4], br[4], cr[4];
        float av[4][CPL];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs),
                                         rb = rsrc((const char*)p.b + xo + r0 * rs),
                                         ra = rsrc(ab + r0 * as);
            RW ar[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs));
                xr[r].template load<kFwdLoad>(rx, o);
                br[r].template load<kFwdLoad>(rb, o);
                if constexpr (PK == 1) ar[r].template load<kFwdLoad>(ra, o);
            }
            if constexpr (PK > 1) {
                float az[4];
                decay_rows_packed<IO, CPL, kFwdDecay>(ra, aoffp, (uint32_t)as, tr0, 0, p.T, p.T, sig_a, az, av);
            } else {
                decay_rows<IO, CPL>(ar, tr0, 0, p.T, p.T, sig_a, av);   // 1 past the end
            }
        }
        float W[4][CPL], G[4][CPL];
        {
            float u[4][CPL];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int m = 0; m < CPL; ++m) u[r][m] = xr[r].get(m) * pregate(br[r].get(m), sig_b);
            chan_scan_fwd<CPL>(av, u, W, G, grp, lane);
        }
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_wl[tw][vch + m] = W[3][m];
                s_cc[tw][vch + m] = G[3][m];
            }
        }
        if constexpr (PARK) {   // (read back by the same lane)
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                s_WG[tw][m][lane] = f32x4{W[0][m], W[1][m], W[2][m], W[3][m]};
                s_WG[tw][CPL + m][lane] = f32x4{G[0][m], G[1][m], G[2][m], G[3][m]};
            }
        }
        {   // c is needed for the outputs only: its loads land during the look-back
            const __amdgpu_buffer_rsrc_t rc = rsrc((const char*)p.c + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                cr[r].template load<kFwdLoad>(rc, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)));
        }
        lds_barrier();

        // ---- wave 0: the chunk's aggregate, the look-back, the inclusive state -----
        if (tw == 0) {
            float V[CPL], P[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) { V[m] = 0.f; P[m] = 1.0f; }
#pragma unroll 1
            for (int r = 0; r < TW; ++r) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float c_ = s_cc[r][vch + m];
                    V[m] = __builtin_fmaf(c_, V[m], s_wl[r][vch + m]);
                    P[m] *= c_;
                }
            }
            float pre[CPL], I[CPL];
            const int64_t so = hb * geo.Dr + geo.coff;   // the virtual head's slice of [B][H][D] states
            chain_link<CPL, Q, 2, kPChannel>(p, seq * nch, ch, nch, V, P, p.h0 ? p.h0 + so : nullptr, lane, grp, n,
                                             pre, I);
            if (grp == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_pre[vch + m] = pre[m];
            }
            store_row<IoF32, CPL>(rsrc(p.h_last ? p.h_last + so : p.chain_incl),
                                  in_range(p.h_last && ch == nch - 1 && grp == 0, vch * 4u), I);
        }
        lds_barrier();

        // ---- outputs: the state entering this wave's sub-block, y, block carriers -----
        float e[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) e[m] = s_pre[vch + m];
#pragma unroll 1
        for (int r = 0; r < tw; ++r) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) e[m] = __builtin_fmaf(s_cc[r][vch + m], e[m], s_wl[r][vch + m]);
        }
        if constexpr (PARK) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const f32x4 w4 = s_WG[tw][m][lane], g4 = s_WG[tw][CPL + m][lane];
#pragma unroll
                for (int r = 0; r < 4; ++r) { W[r][m] = w4[r]; G[r][m] = g4[r]; }
            }
        }
        const __amdgpu_buffer_rsrc_t ry = rsrc((char*)p.y + xo + r0 * rs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                yv[m] = cr[r].get(m) * __builtin_fmaf(G[r][m], e[m], W[r][m]);
                if (p.residual) yv[m] += xr[r].get(m);
            }
            store_row<IO, CPL, kFwdStore>(ry, in_range(tr0 + r < p.T, loff + (uint32_t)(r * rs)), yv);
        }
        // the exact state at the end of a block that ends with this sub-block
        // (a block longer than a chunk that the sequence's end cuts short ends in the last chunk)
        if (p.carriers && (((ch * TW + tw) & smask) == smask || (ch == nch - 1 && tw == TW - 1))) {
            const int64_t blk = r0 >> p.lshift;
            float v[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) v[m] = __builtin_fmaf(s_cc[tw][vch + m], e[m], s_wl[tw][vch + m]);
            store_row<IoF32, CPL>(rsrc(p.carriers + hb * p.nblocks * geo.Dr),
                                  in_range(grp == 0 && geo.ok && blk < p.nblocks, geo.off(p.nblocks, blk) * 4u), v);
        }
        ticket = grab();
    }
}

// The exact recurrence's backward in one pass (mirror of the forward above):
// the chunks are taken from each sequence's end, chain index ci = nch - 1 -
// chunk.  A chunk's aggregate is the adjoint its first token sends towards
// the previous one when nothing enters from its end (the reverse local solve
// D = L^T dh, dh = c * dy, composed over the sub-blocks) and its decay
// product; the value entering a chunk is the adjoint entering from its end
// (dh_last for the last chunk).  The forward states come from the exact
// block carriers (h0 before the first block), as in the three-stage
// backward, and the gradients of a token are those of Sec. 4.2.2 without the
// window's truncation term:  du = D + R eps_in,  dx = b du,  db = x du,
// dc = dy h,  da = sum over channels of h_{t-1} du.
// Lanes of 4 channels park both local solutions in LDS through the
// look-back (64 KB a workgroup), to fit two workgroups a compute unit.  (The
// launcher takes lanes of up to 4 channels: with 8, the kernel needs more
// than 256 registers and measured slower than the three stages.)
template <int CPL>
constexpr bool chain_bwd_park() { return CPL >= 4; }

template <class IO, int CPL, bool FEAT, int Q>
__global__ __launch_bounds__(kChainTW * 64, (CPL == 4 ? 4 : 1)) void swr_bwd_chain_kernel(Params p) {
    constexpr int TW = kChainTW;
    constexpr int TOK = kChainTok;
    constexpr int D = CPL * SB;
    constexpr int ES = IO::ES;
    constexpr bool PARK = chain_bwd_park<CPL>();
    using RW = Row<IO, CPL>;
    const int sig_a = FEAT ? p.sig_a : 0, sig_b = FEAT ? p.sig_b : 0;
    __shared__ float s_wl[TW][D];   // last row of each sub-block's local solve L u
    __shared__ float s_df[TW][D];   // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_c[TW];       // decay product of each sub-block
    __shared__ float s_eps[D];      // the adjoint entering the chunk from its end
    __shared__ f32x4 s_W[PARK ? TW : 1][PARK ? 2 * CPL : 1][PARK ? 64 : 1];   // PARK: W and Dl of each lane
    __shared__ int64_t s_ticket[2];

    const Lanes ln = lanes();
    const int lane = ln.lane, tw = ln.wv, grp = ln.grp, n = ln.n;
    const int64_t S = p.B * p.H, nch = p.nruns, N = S * nch;
    const int64_t rs = p.sx_t * ES, as = p.sa_t * ES, das = p.sa_t * 4;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const uint32_t daoff = (uint32_t)(4 * grp) * (uint32_t)das;
    const uint32_t vch = (uint32_t)(n * CPL);
    const int base = lane & 48;   // first lane of this 16-lane row

    int par = 0;
    auto grab = [&]() {
        if (threadIdx.x == 0) s_ticket[par] = atomicAdd(p.chain_ctr, 1);
        lds_barrier();
        const int64_t t = s_ticket[par];
        par ^= 1;
        return t;
    };
    int64_t ticket = grab();
    for (;;) {
        if (ticket >= N) break;
        const int64_t seq = ticket % S, ci = ticket / S;   // chunk-major from the sequences' ends
        const int64_t ch = nch - 1 - ci;
        const int64_t xo = (seq / p.H * p.sx_b + seq % p.H * p.sx_h) * ES;
        const int64_t ao = seq / p.H * p.sa_b + seq % p.H * p.sa_h;
        const int64_t t0 = ch * TOK, r0 = t0 + tw * SB, tr0 = r0 + 4 * grp;
        // the rows' offsets, recomputed every chunk (an add each) rather than
        // kept across the loop, which spilled registers: an empty asm hides
        // that lo equals loff
        uint32_t lo = loff, dao = daoff, ao_ = aoff;
        asm volatile("" : "+v"(lo), "+v"(dao), "+v"(ao_));

        // ---- loads -------------------------------------------------------------------
        RW xr[4], br[4], cr[4], dyr[4];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc((const char*)p.x + xo + r0 * rs),
                                         rb = rsrc((const char*)p.b + xo + r0 * rs),
                                         rc = rsrc((const char*)p.c + xo + r0 * rs),
                                         rdy = rsrc((const char*)p.dy + xo + r0 * rs);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t o = in_range(tr0 + r < p.T, lo + (uint32_t)(r * rs));
                xr[r].template load<kBwdLoad>(rx, o);
                br[r].template load<kBwdLoad>(rb, o);
                cr[r].template load<kBwdLoad>(rc, o);
                dyr[r].template load<kBwdLoad>(rdy, o);
            }
        }
        const bool a_ok = r0 + n < p.T;
        float a_n = load_scalar<IO, kBwdDecay>(rsrc((const char*)p.a + ao * ES + r0 * as), in_range(a_ok, ao_));
        float ds_n = 1.0f;   // d a / d(input) of token n: 1, or sigma'(z) for a logit z
        if (sig_a) {
            const SigSlope g = sigmoid_slope(a_n);
            ds_n = g.ds;
            a_n = g.s;
        }
        if (!a_ok) a_n = 1.0f;   // past the end the adjoint entering from the end passes intact

        // ---- local solves: W = L (b x) and Dl = L^T dh ----------------------------------
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
                    d4[q] = dyr[q].get(m) * cr[q].get(m);   // dh = c dy
                }
                W[m] = Contract<IO>::run(A, u);
                Dl[m] = Contract<IO>::run(At, d4);
            }
        }
        const float a0 = shfl(a_n, 0);
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[tw][n * CPL + m] = W[m][3];
        }
        if (grp == 0) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_df[tw][n * CPL + m] = a0 * Dl[m][0];
        }
        if (lane == 63) s_c[tw] = dk.c;
        if constexpr (PARK) {   // (read back by the same lane)
#pragma unroll
            for (int m = 0; m < CPL; ++m) { s_W[tw][m][lane] = W[m]; s_W[tw][CPL + m][lane] = Dl[m]; }
        }
        // the exact state entering the chunk (the carrier of the block before it,
        // or h0): requested now, needed after the look-back
        Row<IoF32, CPL> vr;
        if (t0 == 0)
            vr.load(rsrc(p.h0 ? p.h0 + seq * D : p.carriers), in_range(p.h0 != nullptr, vch * 4u));
        else
            vr.load(rsrc(p.carriers + seq * p.nblocks * D), (uint32_t)(((t0 >> p.lshift) - 1) * D + vch) * 4u);
        lds_barrier();

        // ---- wave 0: the chunk's reverse aggregate, the look-back, dh0 -------------------
        if (tw == 0) {
            float V[CPL], P = 1.0f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) V[m] = 0.f;
#pragma unroll 1
            for (int r = TW - 1; r >= 0; --r) {
                const float c_ = s_c[r];
#pragma unroll
                for (int m = 0; m < CPL; ++m) V[m] = __builtin_fmaf(c_, V[m], s_df[r][n * CPL + m]);
                P *= c_;
            }
            float pre[CPL], I[CPL];
            const float Pv[1] = {P};
            chain_link<CPL, Q, 4, kPChunk>(p, seq * nch, ci, nch, V, Pv, p.dh_last ? p.dh_last + seq * D : nullptr,
                                         lane, grp, n, pre, I);
            if (grp == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) s_eps[vch + m] = pre[m];
            }
            store_row<IoF32, CPL>(rsrc(p.dh0 ? p.dh0 + seq * D : p.chain_incl),
                                  in_range(p.dh0 && ch == 0 && grp == 0, vch * 4u), I);
        }
        lds_barrier();

        // ---- the exact state entering this wave's sub-block, the adjoint entering it from its end
        float ein[CPL], epsin[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { ein[m] = vr.get(m); epsin[m] = s_eps[vch + m]; }
#pragma unroll 1
        for (int r = 0; r < tw; ++r) {
            const float c_ = s_c[r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) ein[m] = __builtin_fmaf(c_, ein[m], s_wl[r][n * CPL + m]);
        }
#pragma unroll 1
        for (int r = TW - 1; r > tw; --r) {
            const float c_ = s_c[r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) epsin[m] = __builtin_fmaf(c_, epsin[m], s_df[r][n * CPL + m]);
        }

        // ---- gradients -------------------------------------------------------------------
        if constexpr (PARK) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) { W[m] = s_W[tw][m][lane]; Dl[m] = s_W[tw][CPL + m][lane]; }
        }
        // H = W + g * e_in: the exact state of each row
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
        float Rr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Rr[r] = shfl(dk.L[r], base + 15);   // r_q = L[15][.] at this lane's rows
        const __amdgpu_buffer_rsrc_t rdx = rsrc((char*)p.dx + xo + r0 * rs), rdb = rsrc((char*)p.db + xo + r0 * rs),
                                     rdc = rsrc((char*)p.dc + xo + r0 * rs), rda = rsrc(p.da + ao + r0 * p.sa_t);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float vdx[CPL], vdb[CPL], vdc[CPL], acc = 0.0f;
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
            const float tot = row_sum(acc) * shfl(ds_n, base + 4 * grp + r);
            const bool ok = tr0 + r < p.T;
            const uint32_t o = in_range(ok, lo + (uint32_t)(r * rs));
            store_row<IO, CPL, kBwdStore>(rdx, o, vdx);
            store_row<IO, CPL, kBwdStore>(rdb, o, vdb);
            store_row<IO, CPL, kBwdStore>(rdc, o, vdc);
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, tot), rda,
                                                  (int)in_range(n == 0 && ok, dao + (uint32_t)(r * das)), 0,
                                                  kBwdStore);
        }
        ticket = grab();
    }
}

// Zeroes the chunk flags and the ticket counters before a launch.
__global__ __launch_bounds__(256) void swr_chain_reset_kernel(int32_t* flags, int64_t n, int32_t* ctr) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) flags[i] = 0;
    if (blockIdx.x == 0 && threadIdx.x < 2) ctr[threadIdx.x] = 0;
}

template <class IO, int CPL, int Q>
hipError_t launch_chain_q(const Params& p, hipStream_t st) {
    const dim3 grid((unsigned)p.nwork), block(kChainTW * 64);
    if (p.sig_a || p.sig_b)
        hipLaunchKernelGGL((swr_fwd_chain_kernel<IO, CPL, true, Q>), grid, block, 0, st, p);
    else
        hipLaunchKernelGGL((swr_fwd_chain_kernel<IO, CPL, false, Q>), grid, block, 0, st, p);
    return hipGetLastError();
}

template <class IO, int CPL>
hipError_t launch_chain_cpl(const Params& p, hipStream_t st) {
    if constexpr (chain_qb<CPL, chain_w_in_lds<IO, CPL>()>() == 2) {
        if (p.nruns < kLongChain) return launch_chain_q<IO, CPL, 2>(p, st);
    }
    return launch_chain_q<IO, CPL, 4>(p, st);
}

template <class IO>
hipError_t launch_chain_io(const Params& p, int cpl, hipStream_t st) {
    switch (cpl) {
        case 1: return launch_chain_cpl<IO, 1>(p, st);
        case 2: return launch_chain_cpl<IO, 2>(p, st);
        case 4: return launch_chain_cpl<IO, 4>(p, st);
        case 8: return launch_chain_cpl<IO, 8>(p, st);
        default: return hipErrorInvalidValue;
    }
}

template <int Q>
hipError_t launch_chain_pair_q(const Params& p, hipStream_t st) {
    const dim3 grid((unsigned)p.nwork), block(kChainTW * 64);
    if (p.sig_a || p.sig_b)
        hipLaunchKernelGGL((swr_fwd_chain_pair_kernel<true, Q>), grid, block, 0, st, p);
    else
        hipLaunchKernelGGL((swr_fwd_chain_pair_kernel<false, Q>), grid, block, 0, st, p);
    return hipGetLastError();
}

template <class IO, int CPL, int PK, int Q>
hipError_t launch_chain_pc_q(const Params& p, hipStream_t st) {
    const dim3 grid((unsigned)p.nwork), block(kChainTW * 64);
    if (p.sig_a || p.sig_b)
        hipLaunchKernelGGL((swr_fwd_chain_pc_kernel<IO, CPL, true, PK, Q>), grid, block, 0, st, p);
    else
        hipLaunchKernelGGL((swr_fwd_chain_pc_kernel<IO, CPL, false, PK, Q>), grid, block, 0, st, p);
    return hipGetLastError();
}

template <class IO, int CPL, int PK>
hipError_t launch_chain_pc_cpl(const Params& p, hipStream_t st) {
    return p.nruns < kLongChain ? launch_chain_pc_q<IO, CPL, PK, 2>(p, st) : launch_chain_pc_q<IO, CPL, PK, 4>(p, st);
}

template <class IO>
hipError_t launch_chain_pc_io(const Params& p, int cpl, hipStream_t st) {
    switch (cpl) {
        case 1: return launch_chain_pc_cpl<IO, 1, 1>(p, st);
        case 2: return launch_chain_pc_cpl<IO, 2, 1>(p, st);
        case 4: return launch_chain_pc_cpl<IO, 4, 1>(p, st);
        default: return hipErrorInvalidValue;
    }
}

template <class IO, int CPL>
hipError_t launch_chain_bwd_cpl(const Params& p, hipStream_t st) {
    const dim3 grid((unsigned)p.nwork), block(kChainTW * 64);
    if (p.sig_a || p.sig_b)
        hipLaunchKernelGGL((swr_bwd_chain_kernel<IO, CPL, true, 4>), grid, block, 0, st, p);
    else
        hipLaunchKernelGGL((swr_bwd_chain_kernel<IO, CPL, false, 4>), grid, block, 0, st, p);
    return hipGetLastError();
}

template <class IO>
hipError_t launch_chain_bwd_io(const Params& p, int cpl, hipStream_t st) {
    switch (cpl) {
        case 1: return launch_chain_bwd_cpl<IO, 1>(p, st);
        case 2: return launch_chain_bwd_cpl<IO, 2>(p, st);
        case 4: return launch_chain_bwd_cpl<IO, 4>(p, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t reset_chain(const Params& p, hipStream_t st, int64_t n) {
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(swr_chain_reset_kernel, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0, st,
                       p.chain_flags, n, p.chain_ctr);
    return hipGetLastError();
}

}  // namespace

int chain_tokens() { return kChainTok; }

hipError_t launch_chain_forward(const Params& p, int dtype, int cpl, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    const int64_t n = p.B * p.Hv * p.nruns;
    hipError_t e = reset_chain(p, st, n);
    if (e != hipSuccess || n == 0) return e;
    return dtype == 1 ? launch_chain_io<IoBf16>(p, cpl, st) : launch_chain_io<IoF32>(p, cpl, st);
}

hipError_t launch_chain_forward_pc(const Params& p, int dtype, int cpl, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    const int64_t n = p.B * p.Hv * p.nruns;
    hipError_t e = reset_chain(p, st, n);
    if (e != hipSuccess || n == 0) return e;
    return dtype == 1 ? launch_chain_pc_io<IoBf16>(p, cpl, st) : launch_chain_pc_io<IoF32>(p, cpl, st);
}

hipError_t launch_chain_forward_pair(const Params& p, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    const int64_t n = p.B * (p.H / 2) * p.nruns;
    hipError_t e = reset_chain(p, st, n);
    if (e != hipSuccess || n == 0) return e;
    return p.nruns < kLongChain ? launch_chain_pair_q<2>(p, st) : launch_chain_pair_q<4>(p, st);
}

hipError_t launch_chain_backward(const Params& p, int dtype, int cpl, void* stream) {
    const hipStream_t st = (hipStream_t)stream;
    const int64_t n = p.B * p.H * p.nruns;
    hipError_t e = reset_chain(p, st, n);
    if (e != hipSuccess || n == 0) return e;
    return dtype == 1 ? launch_chain_bwd_io<IoBf16>(p, cpl, st) : launch_chain_bwd_io<IoF32>(p, cpl, st);
}

}  // namespace swr
