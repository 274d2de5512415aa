// swr_device.h -- device-side building blocks shared by the gfx950 kernels of
// the library (swr_kernels.hip: jagged window, exact recurrence, decoding;
// swr_uniform.hip: uniform window): element types, buffer loads and stores
// with range checks, 16-lane DPP scans, the split-bf16 MFMA contraction of a
// 16 x 16 sub-block operator, the sub-block decay operators and the
// workgroup -> work item mapping.  Internal; included by .hip sources only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swr_launch.h"

namespace swr {
namespace {

constexpr int SB = 16;  // tokens per sub-block = MFMA tile edge
// LDS a forward workgroup may spend on its next-step tiles (the copies pay
// off only while several workgroups still fit on a compute unit).
constexpr int kFwdPrefetchLds = 48 * 1024;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Element types
// ---------------------------------------------------------------------------

struct IoBf16 {
    static constexpr int ES = 2;
    __device__ static float to_f32(uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); }
    __device__ static uint32_t from_f32(float v) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v);   // round to nearest even
    }
};

struct IoF32 {
    static constexpr int ES = 4;
};

// ---------------------------------------------------------------------------
// Buffer access
// ---------------------------------------------------------------------------
//
// Every tensor access is a raw buffer load or store: a scalar resource (base
// address of the rows this wave touches in the current step) plus a 32-bit
// per-lane byte offset.  A lane whose row lies outside the valid token range
// passes an offset past the resource's record count, so the hardware returns
// zeros for the load and drops the store; no branches are needed.

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Cache policy of the streaming tensor loads and stores of the forward and
// backward sweeps (the buffer instructions' cache-policy operand: 0 is the
// default policy, 2 the non-temporal streaming hint).  Measured on MI355X at
// B=8, T=16384, H=16, D=128: the hint on the forward's loads and stores
// takes it from 413 to 372 us; on any of the backward's loads or stores it
// makes the backward slower (783 us -> 803-870 us), so it keeps the default.
// The exact backward's stage I (reads only) takes the hint: 1014 -> 978 us.
#ifndef SWR_FWD_LOAD_POLICY
#define SWR_FWD_LOAD_POLICY 2
#endif
#ifndef SWR_FWD_STORE_POLICY
#define SWR_FWD_STORE_POLICY 2
#endif
#ifndef SWR_BWD_LOAD_POLICY
#define SWR_BWD_LOAD_POLICY 0
#endif
#ifndef SWR_BWD_STORE_POLICY
#define SWR_BWD_STORE_POLICY 0
#endif
#ifndef SWR_FWD_DECAY_POLICY
#define SWR_FWD_DECAY_POLICY SWR_FWD_LOAD_POLICY
#endif
#ifndef SWR_BWD_DECAY_POLICY
#define SWR_BWD_DECAY_POLICY SWR_BWD_LOAD_POLICY
#endif
#ifndef SWR_AGG_LOAD_POLICY
#define SWR_AGG_LOAD_POLICY 2
#endif
constexpr int kAggLoad = SWR_AGG_LOAD_POLICY;     // the exact backward's stage I
constexpr int kFwdDecay = SWR_FWD_DECAY_POLICY;   // loads of a
constexpr int kBwdDecay = SWR_BWD_DECAY_POLICY;
constexpr int kFwdLoad = SWR_FWD_LOAD_POLICY;
constexpr int kFwdStore = SWR_FWD_STORE_POLICY;
constexpr int kBwdLoad = SWR_BWD_LOAD_POLICY;
constexpr int kBwdStore = SWR_BWD_STORE_POLICY;

constexpr int kBufferWord3 = 0x00020000;        // raw buffer, 32-bit data format (gfx9 family)
constexpr int kNumRecords = 0x7fffffff;         // every offset below 2^31 - 1 is in range
constexpr uint32_t kOutOfRange = 0x80000000u;   // an offset the range check rejects

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* p) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, kNumRecords, kBufferWord3);
}

__device__ inline uint32_t in_range(bool ok, uint32_t off) { return ok ? off : kOutOfRange; }

// One lane's CPL consecutive channels of one token row, kept as raw bits.
template <class IO, int CPL>
struct Row {
    static constexpr int BYTES = CPL * IO::ES;
    static constexpr int NWORDS = BYTES >= 4 ? BYTES / 4 : 1;
    uint32_t w[NWORDS];

    __device__ void zero() {
#pragma unroll
        for (int i = 0; i < NWORDS; ++i) w[i] = 0;
    }
    template <int POL = 0>
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
        if constexpr (BYTES == 2) {
            w[0] = (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, POL);
        } else if constexpr (BYTES == 4) {
            w[0] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, POL);
        } else if constexpr (BYTES == 8) {
            const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, POL);
            w[0] = v.x; w[1] = v.y;
        } else {
#pragma unroll
            for (int i = 0; i < BYTES / 16; ++i) {
                const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(off + 16 * i), 0, POL);
                w[4 * i + 0] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
            }
        }
    }
    __device__ float get(int m) const {
        if constexpr (IO::ES == 2) {
            const uint32_t v = w[m >> 1];
            return (m & 1) ? __builtin_bit_cast(float, v & 0xffff0000u)
                           : __builtin_bit_cast(float, v << 16);
        } else {
            return __builtin_bit_cast(float, w[m]);
        }
    }
};

// CPL floats of one lane's row slice converted to the I/O type (bf16: round to
// nearest even), kept as the words a vector store writes.
template <class IO, int CPL>
struct Packed {
    static constexpr int BYTES = CPL * IO::ES;
    uint32_t w[BYTES >= 4 ? BYTES / 4 : 1];
    Packed() = default;
    __device__ explicit Packed(const float (&v)[CPL]) {
        if constexpr (IO::ES == 2) {
            if constexpr (CPL == 1) {
                w[0] = IoBf16::from_f32(v[0]);
            } else {
#pragma unroll
                for (int i = 0; i < CPL / 2; ++i)
                    w[i] = IoBf16::from_f32(v[2 * i]) | (IoBf16::from_f32(v[2 * i + 1]) << 16);
            }
        } else {
#pragma unroll
            for (int i = 0; i < CPL; ++i) w[i] = __builtin_bit_cast(uint32_t, v[i]);
        }
    }
    template <int POL = 0>
    __device__ void store(__amdgpu_buffer_rsrc_t r, uint32_t off) const {
        if constexpr (BYTES == 2) {
            __builtin_amdgcn_raw_buffer_store_b16((short)w[0], r, (int)off, 0, POL);
        } else if constexpr (BYTES == 4) {
            __builtin_amdgcn_raw_buffer_store_b32((int)w[0], r, (int)off, 0, POL);
        } else if constexpr (BYTES == 8) {
            __builtin_amdgcn_raw_buffer_store_b64(i32x2{(int)w[0], (int)w[1]}, r, (int)off, 0, POL);
        } else {
#pragma unroll
            for (int i = 0; i < BYTES / 16; ++i)
                __builtin_amdgcn_raw_buffer_store_b128(
                    i32x4{(int)w[4 * i], (int)w[4 * i + 1], (int)w[4 * i + 2], (int)w[4 * i + 3]}, r,
                    (int)(off + 16 * i), 0, POL);
        }
    }
};

// Packs CPL floats to the I/O type and stores them as one vector.
template <class IO, int CPL, int POL = 0>
__device__ inline void store_row(__amdgpu_buffer_rsrc_t r, uint32_t off, const float (&v)[CPL]) {
    Packed<IO, CPL>(v).template store<POL>(r, off);
}

// Asynchronous copy of one row slice per lane from a buffer straight into
// LDS (no registers are involved): lane i's BYTES land at
// lds + chunk * 64 * CHUNK + i * CHUNK for each CHUNK-sized piece.  An
// out-of-range offset is never relied on to write anything.
template <int BYTES>
struct LdsRow {
    static constexpr int CHUNK = BYTES % 16 == 0 ? 16 : 4;
    static constexpr int NCH = BYTES / CHUNK;
    static constexpr int WORDS = BYTES / 4;          // uint32 per lane
    static constexpr int SLOT_WORDS = WORDS * 64;    // uint32 per row slot of a wave

    template <int POL = 0>
    __device__ static void issue(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t* slot) {
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            auto* dst = (__attribute__((address_space(3))) void*)(slot + ch * 64 * (CHUNK / 4));
            if constexpr (CHUNK == 16)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, off + ch * 16, 0, 0, POL);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 4, off + ch * 4, 0, 0, POL);
        }
    }
    __device__ static void read(const uint32_t* slot, int lane, uint32_t (&w)[WORDS]) {
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            if constexpr (CHUNK == 16) {
                const uint4 v = *(const uint4*)(slot + ch * 256 + lane * 4);
                w[4 * ch + 0] = v.x; w[4 * ch + 1] = v.y; w[4 * ch + 2] = v.z; w[4 * ch + 3] = v.w;
            } else {
                w[ch] = slot[ch * 64 + lane];
            }
        }
    }
};

template <class IO, int POL = 0>
__device__ inline float load_scalar(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    if constexpr (IO::ES == 2)
        return IoBf16::to_f32((uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, POL));
    else
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, POL));
}


// ---------------------------------------------------------------------------
// Featurisation (Phalanx, Sec. 5: sigmoid-bounded decay and key-like pre-gate)
// ---------------------------------------------------------------------------

// Logistic sigmoid 1 / (1 + e^-z); e^-z overflows to +inf for very negative
// z, whose reciprocal is the correct limit 0, so the result is finite for
// every finite z.
__device__ inline float sigmoid(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// The pre-gate value b of a loaded element (a logit when sig is set).
__device__ inline float pregate(float z, int sig) { return sig ? sigmoid(z) : z; }

// sigmoid(z) and its slope from one exponential and one reciprocal:
// with E = e^-z and s = 1 / (1 + E), sigmoid(-z) = E s, so the slope
// sigmoid(z) sigmoid(-z) is E s^2 (0 where E overflows, its limit).
struct SigSlope {
    float s, ds;
};
__device__ inline SigSlope sigmoid_slope(float z) {
    const float E = __expf(-z);
    const float s = __builtin_amdgcn_rcpf(1.0f + E);
    return {s, __builtin_isinf(E) ? 0.0f : (E * s) * s};
}

// The same value, opaque to the compiler: a function of it computed again is
// recomputed rather than kept alive in registers since its first use.
__device__ inline float fresh(float v) {
    asm volatile("" : "+v"(v));
    return v;
}

// ---------------------------------------------------------------------------
// Workgroup barrier
// ---------------------------------------------------------------------------

// The waves of a workgroup exchange data through LDS only (no wave reads what
// another wrote to global memory), so a barrier needs to order LDS accesses
// alone: the release / acquire fences of the local address space wait for
// this wave's LDS operations (lgkmcnt) but not for its global loads and
// stores, so loads issued ahead of the barrier (the next step's inputs) stay
// in flight across it.  (__syncthreads also waits for every global access.)
#ifndef SWR_LDS_BARRIER
#define SWR_LDS_BARRIER 1
#endif
__device__ inline void lds_barrier() {
#if SWR_LDS_BARRIER
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
#else
    __syncthreads();
#endif
}

// ---------------------------------------------------------------------------
// Cross-lane helpers (a DPP "row" is 16 lanes on CDNA)
// ---------------------------------------------------------------------------

constexpr int DPP_ROW_SHL = 0x100;
constexpr int DPP_ROW_SHR = 0x110;
constexpr int DPP_ROW_ROR = 0x120;

// Value of lane (n - s) within the row, or `fill` where that lane is outside the row.
template <int CTRL>
__device__ inline float dpp(float v, float fill) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        __builtin_bit_cast(int, fill), __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}

// Inclusive prefix product over lanes 0..n of each 16-lane row (Kogge-Stone doubling).
__device__ inline float row_prefix_prod(float v) {
    v *= dpp<DPP_ROW_SHR + 1>(v, 1.0f);
    v *= dpp<DPP_ROW_SHR + 2>(v, 1.0f);
    v *= dpp<DPP_ROW_SHR + 4>(v, 1.0f);
    v *= dpp<DPP_ROW_SHR + 8>(v, 1.0f);
    return v;
}

// Inclusive suffix product over lanes n..15 of each 16-lane row.
__device__ inline float row_suffix_prod(float v) {
    v *= dpp<DPP_ROW_SHL + 1>(v, 1.0f);
    v *= dpp<DPP_ROW_SHL + 2>(v, 1.0f);
    v *= dpp<DPP_ROW_SHL + 4>(v, 1.0f);
    v *= dpp<DPP_ROW_SHL + 8>(v, 1.0f);
    return v;
}

// Sum over the 16 lanes of each row, broadcast to all of them.
__device__ inline float row_sum(float v) {
    v += dpp<DPP_ROW_ROR + 8>(v, 0.0f);
    v += dpp<DPP_ROW_ROR + 4>(v, 0.0f);
    v += dpp<DPP_ROW_ROR + 2>(v, 0.0f);
    v += dpp<DPP_ROW_ROR + 1>(v, 0.0f);
    return v;
}

__device__ inline float shfl(float v, int src_lane) { return __shfl(v, src_lane, 64); }

// ---------------------------------------------------------------------------
// MFMA contraction of one 16 x 16 x 16 tile: acc[i][j] = sum_k A[i][k] B[k][j]
// with this lane holding A[n][4*grp + q] and B[4*grp + q][j] for q = 0..3.
// ---------------------------------------------------------------------------

// A operand of a split-bf16 contraction: slots 0..3 hold the high parts,
// slots 4..7 the residuals, of this lane's four A entries.
__device__ inline bf16x8 split_operand_a(const float (&v)[4]) {
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const __bf16 hi = (__bf16)v[q];
        r[q] = hi;
        r[4 + q] = (__bf16)(v[q] - (float)hi);
    }
    return r;
}

// Accumulates sum_k A[i][k] (b_hi + b_lo)[k][j] where A was split by
// split_operand_a: pairing each B value with both A halves gives
// (A_hi + A_lo)(B_hi + B_lo) in two K=32 MFMAs with fp32 accumulation.
__device__ inline f32x4 mfma_split(const bf16x8& a, const float (&bv)[4], f32x4 acc) {
    bf16x8 bh, bl;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const __bf16 hi = (__bf16)bv[q];
        const __bf16 lo = (__bf16)(bv[q] - (float)hi);
        bh[q] = hi; bh[4 + q] = hi;
        bl[q] = lo; bl[4 + q] = lo;
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl, acc, 0, 0, 0);
    return acc;
}

__device__ inline f32x4 mfma_f32(const float (&av)[4], const float (&bv)[4], f32x4 acc) {
#pragma unroll
    for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[q], bv[q], acc, 0, 0, 0);
    return acc;
}

template <class IO>
struct Contract {
    // Operand A prepared once per tile set.
    struct A {
        bf16x8 split;
        float f[4];
    };
    __device__ static A prep(const float (&v)[4]) {
        A a;
        if constexpr (IO::ES == 2) {
            a.split = split_operand_a(v);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) a.f[q] = v[q];
        }
        return a;
    }
    __device__ static f32x4 run(const A& a, const float (&bv)[4]) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (IO::ES == 2)
            return mfma_split(a.split, bv, acc);
        else
            return mfma_f32(a.f, bv, acc);
    }
};

// ---------------------------------------------------------------------------
// Workgroup -> work item
// ---------------------------------------------------------------------------

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own L2.
// Give every XCD a contiguous range of work items, so that the H heads of one
// (batch, run) -- which share the cache lines of the [B, T, H] decay tensor --
// and neighbouring runs land on the same L2.
__device__ inline uint32_t xcd_remap(uint32_t id, uint32_t n) {
    const uint32_t q = n >> 3, rem = n & 7, x = id & 7, j = id >> 3;
    return x < rem ? x * (q + 1) + j : rem * (q + 1) + (x - rem) * q + j;
}

struct Work {
    int64_t b, h, t_begin, t_end, run;
};

// A work item is (batch, group of HW consecutive heads, run); the host makes
// HW divide the head count Hv (heads, or virtual heads of the per-channel
// kernels).  Returns the item of head hw of this workgroup's group.
template <int HW>
__device__ inline Work decode_work(const Params& p, int hw) {
    // nwork < 2^31 (checked on the host), so 32-bit arithmetic suffices.
    const uint32_t wid = xcd_remap(blockIdx.x, (uint32_t)p.nwork);
    const uint32_t G = (uint32_t)p.Hv / HW, nruns = (uint32_t)p.nruns;
    Work wk;
    wk.h = (wid % G) * HW + hw;
    const uint32_t rest = wid / G;
    const int64_t run = rest % nruns;
    wk.b = rest / nruns;
    wk.run = run;
    wk.t_begin = run * p.run_len;
    wk.t_end = min(wk.t_begin + p.run_len, p.T);
    return wk;
}

// Per-lane view of one sub-block's decays: the lane's own a (row n of the
// 16-lane row), the operator entries L[n][4*grp + q], the prefix products
// G[k] = a_0 ... a_k for the lane's four token rows, and c = G[15].
struct Decay {
    float a;        // a of token n of the sub-block
    float L[4];     // L[n][4*grp + q]
    float G[4];     // G[4*grp + r]
    float c;        // product of all 16 decays of the sub-block
};

__device__ inline Decay build_decay(float a_n, int grp, int n) {
    Decay d;
    d.a = a_n;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int k = 4 * grp + q;
        // Column k: ones on and above the diagonal, then a cumulative product
        // down the column, then the strict upper triangle set to zero.
        const float v = row_prefix_prod(n > k ? a_n : 1.0f);
        d.L[q] = n >= k ? v : 0.0f;
    }
    const float g = row_prefix_prod(a_n);
    const int base = (threadIdx.x & 63) & 48;   // first lane of this 16-lane row
#pragma unroll
    for (int r = 0; r < 4; ++r) d.G[r] = shfl(g, base + 4 * grp + r);
    d.c = shfl(g, base + 15);
    return d;
}

// ---------------------------------------------------------------------------
// Addressing
// ---------------------------------------------------------------------------

// Row t of one [B, T, H, D] tensor of this workgroup's (batch, head) sits at
// base + t * rs; a lane adds its own 32-bit offset (its row within the
// sub-block and its channel slice).  Keeping base and t * rs uniform lets
// every access use a scalar base plus one vector register of offset.
struct Lanes {
    int lane, wv, grp, n;
};

__device__ inline Lanes lanes() {
    Lanes L;
    L.lane = threadIdx.x & 63;
    L.wv = __builtin_amdgcn_readfirstlane((int)threadIdx.x) >> 6;   // uniform per wave
    L.grp = L.lane >> 4;
    L.n = L.lane & 15;
    return L;
}

// Operand A of the reverse solve D = L^T dh: this lane holds
// L[4*grp + q][n] = a_{n+1} ... a_{4 grp + q} (1 on the diagonal, 0 below),
// a suffix product along the row, built like the forward operator.
__device__ inline void build_decay_transposed(float a_n, int grp, int n, float (&LT)[4]) {
    const float a_next = dpp<DPP_ROW_SHL + 1>(a_n, 1.0f);   // a of token n+1
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int rho = 4 * grp + q;
        const float v = row_suffix_prod(n < rho ? a_next : 1.0f);
        LT[q] = n <= rho ? v : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Per-channel local solves (a decay per channel, or per packed small head)
// ---------------------------------------------------------------------------

// Forward local solve of one sub-block, per channel:  w_k = a_k w_{k-1} + u_k
// and G_k = a_k G_{k-1} (w_{-1} = 0, G_{-1} = 1) for this lane's tokens
// k = 4*grp + r.  A state is carried through a stretch of tokens by
// s -> G s + w, so stretches compose as (G1, w1) then (G2, w2) =
// (G1 G2, G2 w1 + w2).
// Every multiply-add is one explicit fused operation, so that the same scan
// rounds identically in every kernel it is inlined into (the backward's
// recomputation of a block carrier matches the forward's bit for bit).
template <int CPL>
__device__ inline void chan_scan_fwd(const float (&a)[4][CPL], const float (&u)[4][CPL],
                                     float (&w)[4][CPL], float (&G)[4][CPL], int grp, int lane) {
#pragma unroll
    for (int m = 0; m < CPL; ++m) {
        G[0][m] = a[0][m];
        w[0][m] = u[0][m];
#pragma unroll
        for (int r = 1; r < 4; ++r) {
            G[r][m] = a[r][m] * G[r - 1][m];
            w[r][m] = __builtin_fmaf(a[r][m], w[r - 1][m], u[r][m]);
        }
        // Inclusive scan of the row totals over rows 0..grp.
        float tg = G[3][m], tw = w[3][m];
        float pg = shfl(tg, (lane - 16) & 63), pw = shfl(tw, (lane - 16) & 63);
        if (grp >= 1) { tw = __builtin_fmaf(tg, pw, tw); tg = pg * tg; }
        pg = shfl(tg, (lane - 32) & 63); pw = shfl(tw, (lane - 32) & 63);
        if (grp >= 2) { tw = __builtin_fmaf(tg, pw, tw); tg = pg * tg; }
        // Exclusive: the stretch from the sub-block start to this row.
        pg = shfl(tg, (lane - 16) & 63); pw = shfl(tw, (lane - 16) & 63);
        const float gin = grp >= 1 ? pg : 1.0f, win = grp >= 1 ? pw : 0.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            w[r][m] = __builtin_fmaf(G[r][m], win, w[r][m]);
            G[r][m] *= gin;
        }
    }
}


// The decays of one row slice as floats: the loaded values (through the
// sigmoid when they are logits) for tokens in [t_lo, t_hi), 0 before or after
// that range, and 1 past the end of the sequence, so that a partial last
// block's carrier is the state at its last token.
template <class IO, int CPL>
__device__ inline void decay_rows(const Row<IO, CPL> (&ar)[4], int64_t tr0, int64_t t_lo, int64_t t_hi,
                                  int64_t T, int sig, float (&av)[4][CPL]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int64_t t = tr0 + r;
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            const float z = ar[r].get(m);
            av[r][m] = t >= T ? 1.0f : (t >= t_lo && t < t_hi) ? (sig ? sigmoid(z) : z) : 0.0f;
        }
    }
}

// Where a lane's channels live in the per-channel kernels.  A kernel "head"
// (virtual head) is D = CPL * 16 channels.  With a per-channel decay it is
// one real head or one half of it (2^hshift halves).  With packed heads
// (PK > 1: a decay per token and head, heads of 64 / PK channels stored next
// to each other) it is PK adjacent real heads; lane n then holds channels
// (n % (16/PK)) * CPL ... of real head n / (16/PK).  Small heads are
// processed this way because a lane slice of one such head is only 2 or 4
// bytes, while a lane slice of the packed row is 8 or 16.
template <int PK, int CPL>
struct Geo {
    static constexpr int LPH = 16 / PK;   // lanes per real head when packed
    int64_t head;   // first real head of the virtual head
    int64_t coff;   // first channel of the virtual head within its real head
    int64_t Dr;     // channels of a real head (the row length of carriers and states)
    int lh;         // real head of this lane within the virtual head
    int lch;        // first channel of this lane within its real head
    bool ok;        // the lane holds channels (a virtual head of p.dv < D channels
                    // leaves lanes n >= p.nlane idle)
    __device__ Geo(int64_t vh, const Params& p, int n) {
        constexpr int D = CPL * SB;
        if constexpr (PK > 1) {
            head = vh * PK; coff = 0; Dr = D / PK; lh = n / LPH; lch = (n % LPH) * CPL; ok = true;
        } else {
            head = vh >> p.hshift; coff = (vh & ((1 << p.hshift) - 1)) * (int64_t)p.dv; Dr = p.dh;
            lh = 0; lch = (int)coff + n * CPL; ok = n < p.nlane;
        }
    }
    // Offset (in float32 elements) of this lane's slice of row `row` of a
    // per-head array [B*H][rows][Dr], from the start of the virtual head's first head.
    __device__ uint32_t off(int64_t rows, int64_t row) const {
        return (uint32_t)((lh * rows + row) * Dr + lch);
    }
};

// Decays of one row slice for packed heads: one scalar per lane (its real
// head's decay), with the conventions of decay_rows.
template <class IO, int CPL, int POL>
__device__ inline void decay_rows_packed(__amdgpu_buffer_rsrc_t ra, uint32_t aoff, uint32_t astep, int64_t tr0,
                                         int64_t t_lo, int64_t t_hi, int64_t T, int sig, float (&az)[4],
                                         float (&av)[4][CPL]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int64_t t = tr0 + r;
        const bool ok = t >= t_lo && t < t_hi;
        az[r] = load_scalar<IO, POL>(ra, in_range(ok, aoff + (uint32_t)r * astep));
        const float v = t >= T ? 1.0f : ok ? (sig ? sigmoid(az[r]) : az[r]) : 0.0f;
#pragma unroll
        for (int m = 0; m < CPL; ++m) av[r][m] = v;
    }
}

}  // namespace
}  // namespace swr
