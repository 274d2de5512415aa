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

#include "swr_launch.h"

namespace swr {
namespace {

constexpr int SB = 16;  // tokens per sub-block = MFMA tile edge

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
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
        if constexpr (BYTES == 2) {
            w[0] = (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
        } else if constexpr (BYTES == 4) {
            w[0] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
        } else if constexpr (BYTES == 8) {
            const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
            w[0] = v.x; w[1] = v.y;
        } else {
#pragma unroll
            for (int i = 0; i < BYTES / 16; ++i) {
                const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(off + 16 * i), 0, 0);
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

// Packs CPL floats to the I/O type and stores them as one vector.
template <class IO, int CPL>
__device__ inline void store_row(__amdgpu_buffer_rsrc_t r, uint32_t off, const float (&v)[CPL]) {
    constexpr int BYTES = CPL * IO::ES;
    uint32_t w[BYTES >= 4 ? BYTES / 4 : 1];
    if constexpr (IO::ES == 2) {
        if constexpr (CPL == 1) {
            __builtin_amdgcn_raw_buffer_store_b16((short)IoBf16::from_f32(v[0]), r, (int)off, 0, 0);
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
        __builtin_amdgcn_raw_buffer_store_b32((int)w[0], r, (int)off, 0, 0);
    } else if constexpr (BYTES == 8) {
        __builtin_amdgcn_raw_buffer_store_b64(i32x2{(int)w[0], (int)w[1]}, r, (int)off, 0, 0);
    } else if constexpr (BYTES >= 16) {
#pragma unroll
        for (int i = 0; i < BYTES / 16; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(
                i32x4{(int)w[4 * i], (int)w[4 * i + 1], (int)w[4 * i + 2], (int)w[4 * i + 3]}, r,
                (int)(off + 16 * i), 0, 0);
    }
}

template <class IO>
__device__ inline float load_scalar(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    if constexpr (IO::ES == 2)
        return IoBf16::to_f32((uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0));
    else
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
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
__device__ inline int64_t xcd_remap(int64_t id, int64_t n) {
    const int64_t q = n / 8, rem = n % 8, x = id % 8, j = id / 8;
    return x < rem ? x * (q + 1) + j : rem * (q + 1) + (x - rem) * q + j;
}

struct Work {
    int64_t b, h, t_begin, t_end;
};

__device__ inline Work decode_work(const Params& p) {
    const int64_t wid = xcd_remap(blockIdx.x, p.nwork);
    Work wk;
    wk.h = wid % p.H;
    const int64_t rest = wid / p.H;
    const int64_t run = rest % p.nruns;
    wk.b = rest / p.nruns;
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

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------

template <class IO, int CPL, int NW>
__global__ __launch_bounds__(NW * 64) void swr_fwd_kernel(Params p) {
    constexpr int D = CPL * SB;
    constexpr int STEP = NW * SB;
    constexpr int ES = IO::ES;
    __shared__ float s_wl[2][NW][D];   // last row of each sub-block's local solve
    __shared__ float s_c[2][NW];       // each sub-block's decay product

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const Work wk = decode_work(p);
    const int l = p.block;
    const int S = l / SB;              // sub-blocks per block
    const int64_t t_lo = max(wk.t_begin - (int64_t)l, (int64_t)0);  // first token read
    const int64_t halo = wk.t_begin > 0 ? (l + STEP - 1) / STEP : 0;

    const int64_t xo = (wk.b * p.sx_b + wk.h * p.sx_h) * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    char* yb = (char*)p.y + xo;
    const char* ab = (const char*)p.a + (wk.b * p.sa_b + wk.h * p.sa_h) * ES;
    const int64_t rs = p.sx_t * ES;    // row stride in bytes
    const int64_t as = p.sa_t * ES;
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CPL * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;

    float e[CPL], s[CPL];   // carriers at the start of the step: full and block-restarted
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }

    int buf = 0;
    for (int64_t t0 = wk.t_begin - halo * STEP; t0 < wk.t_end; t0 += STEP, buf ^= 1) {
        const int64_t r0 = t0 + wv * SB;          // first token of this wave's sub-block (uniform)
        const int64_t tr0 = r0 + 4 * grp;         // first of this lane's four tokens

        // ---- loads -------------------------------------------------------
        const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs),
                                     rc = rsrc(cb + r0 * rs), ry = rsrc(yb + r0 * rs);
        Row<IO, CPL> xr[4], br[4], cr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            const uint32_t o = loff + (uint32_t)(r * rs);
            const uint32_t ox = in_range(t >= t_lo && t < wk.t_end, o);
            xr[r].load(rx, ox);
            br[r].load(rb, ox);
            cr[r].load(rc, in_range(t >= wk.t_begin && t < wk.t_end, o));
        }
        const int64_t ta = r0 + n;
        const float a_n = load_scalar<IO>(rsrc(ab + r0 * as), in_range(ta >= t_lo && ta < wk.t_end, aoff));

        // ---- local solve W = L U on the matrix cores ---------------------
        const Decay dk = build_decay(a_n, grp, n);
        const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
        f32x4 W[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            float u[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * br[q].get(m);   // pre-gate b*x
            W[m] = Contract<IO>::run(A, u);
        }

        // ---- carriers through LDS ------------------------------------------
        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[buf][wv][n * CPL + m] = W[m][3];
        }
        if (lane == 63) s_c[buf][wv] = dk.c;
        __syncthreads();

        float ein[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) ein[m] = 0.f;
        for (int r = 0; r < NW; ++r) {
            if (r % S == 0) {   // a block starts: its carry-in is the previous block's v
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
            }
            if (r == wv) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) ein[m] = e[m];
            }
            const float cr_ = s_c[buf][r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float wl = s_wl[buf][r][n * CPL + m];
                e[m] = cr_ * e[m] + wl;
                s[m] = cr_ * s[m] + wl;
            }
        }

        // ---- rank-one injection, read-out gate, store ----------------------
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float yv[CPL];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float hv = W[m][r] + dk.G[r] * ein[m];
                yv[m] = cr[r].get(m) * hv;
                if (p.residual) yv[m] += xr[r].get(m);
            }
            store_row<IO, CPL>(ry, in_range(t >= wk.t_begin && t < wk.t_end, loff + (uint32_t)(r * rs)), yv);
        }
    }
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------

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

// Gradient of the truncated forward.  du = L~^T dh with dh = c * dy is itself a
// block two-pass run backwards: du_t = L_t^T dh_t + r_t C_{t+1}, where
// r_t = e_l^T L_t and C_{t+1} = g_{t+1}^T dh_{t+1} comes from the next block.
// The decay gradient of token k (block t) collects, over the channels, the
// state entering step k times the adjoint leaving it, for the two windows
// that contain k:  da_k = sum_mu [ w_{t,k-1} du_k + g_{t,k-1} v_{t-1} D_{t,k} ]
// with w the block-restarted local state, D_t = L_t^T dh_t and v_{t-1} the
// previous block's carrier (w_{t,-1} = 0, g_{t,-1} = 1).
//
// Register budget: the step's look-ahead tiles (c, dy of the next step) are
// handed to the next step through a wave-private LDS slot (two slots used in
// turn), and the epilogue runs over the channels in NPASS passes, each
// recomputing its part of W = L u and D = L^T dh on the matrix cores, so that
// only one pass's accumulators are live at a time.  In pass ps lane n owns
// channels ps*16*CH + n*CH .. + CH-1, so every load and store instruction
// covers 16*CH contiguous channels of a row (whole memory sectors).
template <class IO, int CPL, int NW>
struct BwdShape {
    static constexpr int NPASS = CPL >= 4 ? 2 : 1;      // epilogue passes
    static constexpr int CH = CPL / NPASS;               // channels per lane per pass
    static constexpr int HWD = Row<IO, CH>::NWORDS;      // words of one lane's pass slice
    static constexpr int NWD = NPASS * HWD;
    static constexpr int HAND_BYTES = 2 * NW * 2 * 4 * NWD * 64 * 4;
    // Hand over through LDS when both slots fit beside the carrier buffers;
    // otherwise the next step re-reads c and dy from global memory.
    static constexpr bool HAND_LDS = HAND_BYTES <= 128 * 1024;
};

template <class IO, int CPL, int NW>
__global__ __launch_bounds__(NW * 64) void swr_bwd_kernel(Params p) {
    constexpr int D = CPL * SB;
    constexpr int STEP = NW * SB;
    constexpr int ES = IO::ES;
    using Sh = BwdShape<IO, CPL, NW>;
    using RH = Row<IO, Sh::CH>;
    constexpr int NPASS = Sh::NPASS, CH = Sh::CH, HWD = Sh::HWD, NWD = Sh::NWD;
    constexpr int PIECE = 16 * CH;                       // channels covered by one pass
    __shared__ float s_wl[2][NW][D];    // last row of each sub-block's local solve
    __shared__ float s_c[2][NW];        // decay product of each sub-block
    __shared__ float s_df[3][NW][D];    // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_cf[3][NW];       // decay products for the reverse carriers
    // Wave-private hand-over of the look-ahead's c and dy tiles: [slot][wave][c|dy][row][word][lane].
    __shared__ uint32_t s_hand[Sh::HAND_LDS ? 2 : 1][Sh::HAND_LDS ? NW : 1][2][4][NWD][64];

    const Lanes ln = lanes();
    const int lane = ln.lane, wv = ln.wv, grp = ln.grp, n = ln.n;
    const Work wk = decode_work(p);
    const int l = p.block;
    const int S = l / SB;
    const int64_t t_lo = max(wk.t_begin - (int64_t)l, (int64_t)0);
    const int64_t t_la = min(wk.t_end + (int64_t)l, p.T);   // end (excl.) of the look-ahead

    const int64_t xo = (wk.b * p.sx_b + wk.h * p.sx_h) * ES;
    const char* xb = (const char*)p.x + xo;
    const char* bb = (const char*)p.b + xo;
    const char* cb = (const char*)p.c + xo;
    const char* dyb = (const char*)p.dy + xo;
    char* dxb = (char*)p.dx + xo;
    char* dbb = (char*)p.db + xo;
    char* dcb = (char*)p.dc + xo;
    const int64_t ao = wk.b * p.sa_b + wk.h * p.sa_h;
    const char* ab = (const char*)p.a + ao * ES;
    char* dab = (char*)(p.da + ao);
    const int64_t rs = p.sx_t * ES;
    const int64_t as = p.sa_t * ES;
    const int64_t das = p.sa_t * 4;
    // Byte offset of this lane's slice in pass 0 of row 4*grp; pass ps adds ps*PIECE channels.
    const uint32_t loff = (uint32_t)(4 * grp) * (uint32_t)rs + (uint32_t)(n * CH * ES);
    const uint32_t aoff = (uint32_t)n * (uint32_t)as;
    const uint32_t daoff = (uint32_t)(4 * grp) * (uint32_t)das;
    const int base = lane & 48;   // first lane of this 16-lane row
    auto chan = [&](int ps, int j) { return ps * PIECE + n * CH + j; };   // channel of slot (ps, j)

    float e[CPL], s[CPL];   // forward carriers at the step start (full, block-restarted)
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }

    // The sweep starts one step early (the halo step): it recovers the forward
    // carrier entering the run and the look-ahead for the run's first step.
    int k = 0;
    for (int64_t t0 = wk.t_begin - STEP; t0 < wk.t_end; t0 += STEP, ++k) {
        const int bw = k & 1, bc = k % 3, bn = (k + 1) % 3;
        const int hs = Sh::HAND_LDS ? (k & 1) : 0;          // slot holding this step's c, dy
        const int64_t r0 = t0 + wv * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const bool out_step = t0 >= wk.t_begin;

        // ---- loads: this step's x, b, a and the next step's c, dy, a ---------
        RH xr[NPASS][4], br[NPASS][4];
        {
            const __amdgpu_buffer_rsrc_t rx = rsrc(xb + r0 * rs), rb = rsrc(bb + r0 * rs);
            const __amdgpu_buffer_rsrc_t rcn = rsrc(cb + (r0 + STEP) * rs), rdyn = rsrc(dyb + (r0 + STEP) * rs);
            RH cn[NPASS][4], dyn[NPASS][4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = tr0 + r, tn = t + STEP;
                const bool okx = t >= t_lo && t < wk.t_end;
                const bool okn = tn >= wk.t_begin && tn < t_la;
#pragma unroll
                for (int ps = 0; ps < NPASS; ++ps) {
                    const uint32_t o = loff + (uint32_t)(r * rs + ps * PIECE * ES);
                    xr[ps][r].load(rx, in_range(okx, o));
                    br[ps][r].load(rb, in_range(okx, o));
                    cn[ps][r].load(rcn, in_range(okn, o));
                    dyn[ps][r].load(rdyn, in_range(okn, o));
                }
            }
            const int64_t tan_ = r0 + n + STEP;
            const float a_nn = load_scalar<IO>(rsrc(ab + (r0 + STEP) * as),
                                               in_range(tan_ >= wk.t_begin && tan_ < t_la, aoff));

            // ---- look-ahead: first row of the next step's reverse solve ------
            // It feeds the reverse carrier entering this step's last block.
            float LT[4];
            build_decay_transposed(a_nn, grp, n, LT);
            const typename Contract<IO>::A At = Contract<IO>::prep(LT);
            const float cn_ = shfl(row_prefix_prod(a_nn), 15);
            const float a0 = shfl(a_nn, 0);
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
                for (int j = 0; j < CH; ++j) {
                    float dh[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) dh[q] = dyn[ps][q].get(j) * cn[ps][q].get(j);
                    const f32x4 Dn = Contract<IO>::run(At, dh);
                    if (grp == 0) s_df[bn][wv][chan(ps, j)] = a0 * Dn[0];
                }
            if (lane == 0) s_cf[bn][wv] = cn_;
            if constexpr (Sh::HAND_LDS) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
                        for (int i = 0; i < HWD; ++i) {
                            s_hand[hs ^ 1][wv][0][r][ps * HWD + i][lane] = cn[ps][r].w[i];
                            s_hand[hs ^ 1][wv][1][r][ps * HWD + i][lane] = dyn[ps][r].w[i];
                        }
            }
        }
        const int64_t ta = r0 + n;
        const float a_n = load_scalar<IO>(rsrc(ab + r0 * as), in_range(ta >= t_lo && ta < wk.t_end, aoff));

        // ---- forward recompute: last local row W[15] of each channel ---------
        const Decay dk = build_decay(a_n, grp, n);
        const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[ps][q].get(j) * br[ps][q].get(j);
                const f32x4 W = Contract<IO>::run(A, u);
                if (grp == 3) s_wl[bw][wv][chan(ps, j)] = W[3];
            }
        if (lane == 63) s_c[bw][wv] = dk.c;
        __syncthreads();

        if (!out_step) {
            // Halo step: only advance the forward carriers.
#pragma unroll 1
            for (int r = 0; r < NW; ++r) {
                if (r % S == 0) {
#pragma unroll
                    for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
                }
                const float c_ = s_c[bw][r];
#pragma unroll
                for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
                    for (int j = 0; j < CH; ++j) {
                        const float wl = s_wl[bw][r][chan(ps, j)];
                        e[ps * CH + j] = c_ * e[ps * CH + j] + wl;
                        s[ps * CH + j] = c_ * s[ps * CH + j] + wl;
                    }
            }
            continue;
        }

        // ---- per-step constants of the epilogue -----------------------------
        float LTc[4];
        build_decay_transposed(a_n, grp, n, LTc);
        const typename Contract<IO>::A Atc = Contract<IO>::prep(LTc);
        float Rr[4], Gsh[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Rr[r] = shfl(dk.L[r], base + 15);   // r_q = L[15][.] at this lane's rows
        {
            const float gprev = shfl(dk.G[3], (lane - 16) & 63);      // G[k-1], G[-1] = 1
            Gsh[0] = grp == 0 ? 1.0f : gprev;
            Gsh[1] = dk.G[0]; Gsh[2] = dk.G[1]; Gsh[3] = dk.G[2];
        }
        float da_acc[4] = {0.f, 0.f, 0.f, 0.f};
        const __amdgpu_buffer_rsrc_t rdx = rsrc(dxb + r0 * rs), rdb = rsrc(dbb + r0 * rs),
                                     rdc = rsrc(dcb + r0 * rs);

#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps) {
            const int m0 = ps * CH;
            // c and dy of this step for the pass's channels.
            RH cr[4], dyr[4];
            if constexpr (Sh::HAND_LDS) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int i = 0; i < HWD; ++i) {
                        cr[r].w[i] = s_hand[hs][wv][0][r][ps * HWD + i][lane];
                        dyr[r].w[i] = s_hand[hs][wv][1][r][ps * HWD + i][lane];
                    }
            } else {
                const __amdgpu_buffer_rsrc_t rc = rsrc(cb + r0 * rs), rdy = rsrc(dyb + r0 * rs);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const uint32_t o = in_range(tr0 + r < wk.t_end, loff + (uint32_t)(r * rs + ps * PIECE * ES));
                    cr[r].load(rc, o);
                    dyr[r].load(rdy, o);
                }
            }

            // Forward carriers entering this wave's sub-block, and their update.
            float ein[CH], sin_[CH];
#pragma unroll
            for (int j = 0; j < CH; ++j) { ein[j] = 0.f; sin_[j] = 0.f; }
#pragma unroll 1
            for (int r = 0; r < NW; ++r) {
                if (r % S == 0) {
#pragma unroll
                    for (int j = 0; j < CH; ++j) { e[m0 + j] = s[m0 + j]; s[m0 + j] = 0.f; }
                }
                if (r == wv) {
#pragma unroll
                    for (int j = 0; j < CH; ++j) { ein[j] = e[m0 + j]; sin_[j] = s[m0 + j]; }
                }
                const float c_ = s_c[bw][r];
#pragma unroll
                for (int j = 0; j < CH; ++j) {
                    const float wl = s_wl[bw][r][chan(ps, j)];
                    e[m0 + j] = c_ * e[m0 + j] + wl;
                    s[m0 + j] = c_ * s[m0 + j] + wl;
                }
            }
            // Reverse carriers: from the end of the next step's first block back
            // to this wave's sub-block.  eps is the full adjoint entering a
            // sub-block from the right, pr the one restarted at its block's end.
            float eps[CH], pr[CH];
#pragma unroll
            for (int j = 0; j < CH; ++j) { eps[j] = 0.f; pr[j] = 0.f; }
#pragma unroll 1
            for (int r = S - 1; r >= 0; --r) {
                const float c_ = s_cf[bn][r];
#pragma unroll
                for (int j = 0; j < CH; ++j) pr[j] = c_ * pr[j] + s_df[bn][r][chan(ps, j)];
            }
#pragma unroll 1
            for (int r = NW - 1; r >= wv; --r) {
                if (r % S == S - 1) {
#pragma unroll
                    for (int j = 0; j < CH; ++j) { eps[j] = pr[j]; pr[j] = 0.f; }
                }
                if (r > wv) {
                    const float c_ = s_cf[bc][r];
#pragma unroll
                    for (int j = 0; j < CH; ++j) {
                        const float df = s_df[bc][r][chan(ps, j)];
                        eps[j] = c_ * eps[j] + df;
                        pr[j] = c_ * pr[j] + df;
                    }
                }
            }

            // Recompute this pass's tiles: W = L (b*x) and D = L^T (c*dy).
            f32x4 W[CH], Dl[CH];
            float wup[CH];   // local state of the row above this lane's first row (0 above row 0)
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                float u[4], dh[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    u[q] = xr[ps][q].get(j) * br[ps][q].get(j);
                    dh[q] = dyr[q].get(j) * cr[q].get(j);
                }
                W[j] = Contract<IO>::run(A, u);
                Dl[j] = Contract<IO>::run(Atc, dh);
                const float v = shfl(W[j][3], (lane - 16) & 63);
                wup[j] = grp == 0 ? 0.0f : v;
            }

#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = tr0 + r;
                float vdx[CH], vdb[CH], vdc[CH];
                float acc = 0.f, acc2 = 0.f;
#pragma unroll
                for (int j = 0; j < CH; ++j) {
                    const float hv = W[j][r] + dk.G[r] * ein[j];           // jagged-window state
                    const float dyv = dyr[r].get(j);
                    vdc[j] = dyv * hv;
                    const float du = Dl[j][r] + Rr[r] * eps[j];            // adjoint of u
                    const float dblk = Dl[j][r] + Rr[r] * pr[j];           // ... from this block's rows
                    vdx[j] = br[ps][r].get(j) * du;
                    if (p.residual) vdx[j] += dyv;
                    vdb[j] = xr[ps][r].get(j) * du;
                    const float wprev = r == 0 ? wup[j] : W[j][r - 1];
                    acc += wprev * du;
                    acc2 += sin_[j] * du + (ein[j] - sin_[j]) * dblk;
                }
                da_acc[r] += acc + Gsh[r] * acc2;
                const uint32_t o = in_range(t >= wk.t_begin && t < wk.t_end,
                                            loff + (uint32_t)(r * rs + ps * PIECE * ES));
                store_row<IO, CH>(rdx, o, vdx);
                store_row<IO, CH>(rdb, o, vdb);
                store_row<IO, CH>(rdc, o, vdc);
            }
        }
        const __amdgpu_buffer_rsrc_t rda = rsrc(dab + r0 * das);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float tot = row_sum(da_acc[r]);
            const int64_t t = tr0 + r;
            __builtin_amdgcn_raw_buffer_store_b32(
                __builtin_bit_cast(int, tot), rda,
                (int)in_range(n == 0 && t >= wk.t_begin && t < wk.t_end, daoff + (uint32_t)(r * das)), 0, 0);
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

template <class IO, int CPL, int NW>
static hipError_t launch_one(const Params& p, bool backward, hipStream_t stream) {
    const dim3 grid((unsigned)p.nwork), block(NW * 64);
    if (backward)
        hipLaunchKernelGGL((swr_bwd_kernel<IO, CPL, NW>), grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL((swr_fwd_kernel<IO, CPL, NW>), grid, block, 0, stream, p);
    return hipGetLastError();
}

template <class IO, int CPL>
static hipError_t launch_nw(const Params& p, int nw, bool backward, hipStream_t stream) {
    if (nw == 4) return launch_one<IO, CPL, 4>(p, backward, stream);
    if (nw == 8) return launch_one<IO, CPL, 8>(p, backward, stream);
    return hipErrorInvalidValue;
}

template <class IO>
static hipError_t launch_cpl(const Params& p, int D, int nw, bool backward, hipStream_t stream) {
    switch (D) {
        case 16: return launch_nw<IO, 1>(p, nw, backward, stream);
        case 32: return launch_nw<IO, 2>(p, nw, backward, stream);
        case 64: return launch_nw<IO, 4>(p, nw, backward, stream);
        case 128: return launch_nw<IO, 8>(p, nw, backward, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch(const Params& p, int dtype, int D, int nw, bool backward, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    if (dtype == 1) return launch_cpl<IoBf16>(p, D, nw, backward, st);
    return launch_cpl<IoF32>(p, D, nw, backward, st);
}

}  // namespace swr
