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
    __device__ void load(const void* p) {
        if constexpr (BYTES == 2) {
            w[0] = *(const uint16_t*)p;
        } else if constexpr (BYTES == 4) {
            w[0] = *(const uint32_t*)p;
        } else if constexpr (BYTES == 8) {
            uint2 v = *(const uint2*)p;
            w[0] = v.x; w[1] = v.y;
        } else {
#pragma unroll
            for (int i = 0; i < BYTES / 16; ++i) {
                uint4 v = ((const uint4*)p)[i];
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
__device__ inline void store_row(void* p, const float (&v)[CPL]) {
    if constexpr (IO::ES == 2) {
        if constexpr (CPL == 1) {
            *(uint16_t*)p = (uint16_t)IoBf16::from_f32(v[0]);
        } else {
            uint32_t w[CPL / 2];
#pragma unroll
            for (int i = 0; i < CPL / 2; ++i)
                w[i] = IoBf16::from_f32(v[2 * i]) | (IoBf16::from_f32(v[2 * i + 1]) << 16);
            if constexpr (CPL == 2) {
                *(uint32_t*)p = w[0];
            } else if constexpr (CPL == 4) {
                *(uint2*)p = make_uint2(w[0], w[1]);
            } else {
                *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
    } else {
        if constexpr (CPL == 1) {
            *(float*)p = v[0];
        } else if constexpr (CPL == 2) {
            *(float2*)p = make_float2(v[0], v[1]);
        } else {
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i)
                ((float4*)p)[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
        }
    }
}

template <class IO>
__device__ inline float load_scalar(const void* p) {
    if constexpr (IO::ES == 2)
        return IoBf16::to_f32(*(const uint16_t*)p);
    else
        return *(const float*)p;
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
// Forward
// ---------------------------------------------------------------------------

template <class IO, int CPL, int NW>
__global__ __launch_bounds__(NW * 64) void swr_fwd_kernel(Params p) {
    constexpr int D = CPL * SB;
    constexpr int STEP = NW * SB;
    __shared__ float s_wl[2][NW][D];   // last row of each sub-block's local solve
    __shared__ float s_c[2][NW];       // each sub-block's decay product

    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int grp = lane >> 4, n = lane & 15;
    const Work wk = decode_work(p);
    const int l = p.block;
    const int S = l / SB;              // sub-blocks per block
    const int64_t t_lo = max(wk.t_begin - (int64_t)l, (int64_t)0);  // first token read
    const int64_t halo = wk.t_begin > 0 ? (l + STEP - 1) / STEP : 0;

    const char* xp = (const char*)p.x + (wk.b * p.sx_b + wk.h * p.sx_h + n * CPL) * IO::ES;
    const char* bp = (const char*)p.b + (wk.b * p.sx_b + wk.h * p.sx_h + n * CPL) * IO::ES;
    const char* cp = (const char*)p.c + (wk.b * p.sx_b + wk.h * p.sx_h + n * CPL) * IO::ES;
    char* yp = (char*)p.y + (wk.b * p.sx_b + wk.h * p.sx_h + n * CPL) * IO::ES;
    const char* ap = (const char*)p.a + (wk.b * p.sa_b + wk.h * p.sa_h) * IO::ES;
    const int64_t rs = p.sx_t * IO::ES;   // row stride in bytes

    float e[CPL], s[CPL];   // carriers at the start of the step: full and block-restarted
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }

    int buf = 0;
    for (int64_t t0 = wk.t_begin - halo * STEP; t0 < wk.t_end; t0 += STEP, buf ^= 1) {
        const int64_t r0 = t0 + wv * SB;          // first token of this wave's sub-block
        const int64_t tr0 = r0 + 4 * grp;         // first of this lane's four tokens

        // ---- loads -------------------------------------------------------
        Row<IO, CPL> xr[4], br[4], cr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            if (t >= t_lo && t < wk.t_end) {
                xr[r].load(xp + t * rs);
                br[r].load(bp + t * rs);
            } else {
                xr[r].zero(); br[r].zero();
            }
            if (t >= wk.t_begin && t < wk.t_end) cr[r].load(cp + t * rs); else cr[r].zero();
        }
        const int64_t ta = r0 + n;
        const float a_n = (ta >= t_lo && ta < wk.t_end) ? load_scalar<IO>(ap + ta * p.sa_t * IO::ES) : 0.0f;

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
            if (t >= wk.t_begin && t < wk.t_end) {
                float yv[CPL];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float hv = W[m][r] + dk.G[r] * ein[m];
                    yv[m] = cr[r].get(m) * hv;
                    if (p.residual) yv[m] += xr[r].get(m);
                }
                store_row<IO, CPL>(yp + t * rs, yv);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------

template <class IO, int CPL, int NW>
__global__ __launch_bounds__(NW * 64) void swr_bwd_kernel(Params p) {
    constexpr int D = CPL * SB;
    constexpr int STEP = NW * SB;
    __shared__ float s_wl[2][NW][D];    // last row of each sub-block's local solve
    __shared__ float s_c[2][NW];        // decay product of each sub-block
    __shared__ float s_df[3][NW][D];    // a_0 * first row of each sub-block's L^T dh
    __shared__ float s_cf[3][NW];       // decay products for the reverse carriers

    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int grp = lane >> 4, n = lane & 15;
    const Work wk = decode_work(p);
    const int l = p.block;
    const int S = l / SB;
    const int64_t t_lo = max(wk.t_begin - (int64_t)l, (int64_t)0);
    const int64_t t_la = min(wk.t_end + (int64_t)l, p.T);   // last token (excl.) of the look-ahead

    const int64_t off = (wk.b * p.sx_b + wk.h * p.sx_h + n * CPL) * IO::ES;
    const char* xp = (const char*)p.x + off;
    const char* bp = (const char*)p.b + off;
    const char* cp = (const char*)p.c + off;
    const char* dyp = (const char*)p.dy + off;
    char* dxp = (char*)p.dx + off;
    char* dbp = (char*)p.db + off;
    char* dcp = (char*)p.dc + off;
    const char* ap = (const char*)p.a + (wk.b * p.sa_b + wk.h * p.sa_h) * IO::ES;
    float* dap = p.da + (wk.b * p.sa_b + wk.h * p.sa_h);
    const int64_t rs = p.sx_t * IO::ES;
    const int64_t as = p.sa_t * IO::ES;

    float e[CPL], s[CPL];
#pragma unroll
    for (int m = 0; m < CPL; ++m) { e[m] = 0.f; s[m] = 0.f; }

    // The sweep starts one step early (the halo step): it recovers the forward
    // carrier entering the run and the look-ahead of the run's first step.
    int k = 0;
    for (int64_t t0 = wk.t_begin - STEP; t0 < wk.t_end; t0 += STEP, ++k) {
        const int bw = k & 1, bc = k % 3, bn = (k + 1) % 3;
        const int64_t r0 = t0 + wv * SB;
        const int64_t tr0 = r0 + 4 * grp;
        const bool out_step = t0 >= wk.t_begin;

        // ---- loads: this step's x, b, c, dy, a and the next step's c, dy, a --
        Row<IO, CPL> xr[4], br[4], cr[4], dyr[4], cn[4], dyn[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            if (t >= t_lo && t < wk.t_end) {
                xr[r].load(xp + t * rs);
                br[r].load(bp + t * rs);
            } else {
                xr[r].zero(); br[r].zero();
            }
            if (out_step && t >= wk.t_begin && t < wk.t_end) {
                cr[r].load(cp + t * rs);
                dyr[r].load(dyp + t * rs);
            } else {
                cr[r].zero(); dyr[r].zero();
            }
            const int64_t tn = t + STEP;
            if (tn >= wk.t_begin && tn < t_la) {
                cn[r].load(cp + tn * rs);
                dyn[r].load(dyp + tn * rs);
            } else {
                cn[r].zero(); dyn[r].zero();
            }
        }
        const int64_t ta = r0 + n;
        const float a_n = (ta >= t_lo && ta < wk.t_end) ? load_scalar<IO>(ap + ta * as) : 0.0f;
        const int64_t tan_ = ta + STEP;
        const float a_nn = (tan_ >= wk.t_begin && tan_ < t_la) ? load_scalar<IO>(ap + tan_ * as) : 0.0f;

        // ---- look-ahead: reverse local solve of the next step's sub-block ----
        // Only its first row is used here (the reverse carrier entering this
        // step's last block); the full solve is redone when that step comes.
        {
            // A operand: L^T, i.e. this lane holds L[4*grp + q][n] = a_{n+1} ... a_{4 grp + q}.
            const float a_next = dpp<DPP_ROW_SHL + 1>(a_nn, 1.0f);   // a of token n+1
            float LT[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int rho = 4 * grp + q;
                const float v = row_suffix_prod(n < rho ? a_next : 1.0f);
                LT[q] = n <= rho ? v : 0.0f;
            }
            const typename Contract<IO>::A At = Contract<IO>::prep(LT);
            const float cn_ = shfl(row_prefix_prod(a_nn), 15);
            const float a0 = shfl(a_nn, 0);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float dh[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) dh[q] = dyn[q].get(m) * cn[q].get(m);
                const f32x4 Dn = Contract<IO>::run(At, dh);
                if (grp == 0) s_df[bn][wv][n * CPL + m] = a0 * Dn[0];
            }
            if (lane == 0) s_cf[bn][wv] = cn_;
        }

        // ---- this step: forward recompute and reverse local solve -----------
        const Decay dk = build_decay(a_n, grp, n);
        f32x4 W[CPL], Dl[CPL];
        {
            const typename Contract<IO>::A A = Contract<IO>::prep(dk.L);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) u[q] = xr[q].get(m) * br[q].get(m);
                W[m] = Contract<IO>::run(A, u);
            }
        }
        {
            const float a_next = dpp<DPP_ROW_SHL + 1>(a_n, 1.0f);
            float LT[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int rho = 4 * grp + q;
                const float v = row_suffix_prod(n < rho ? a_next : 1.0f);
                LT[q] = n <= rho ? v : 0.0f;
            }
            const typename Contract<IO>::A At = Contract<IO>::prep(LT);
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                float dh[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) dh[q] = dyr[q].get(m) * cr[q].get(m);   // dh = dy * c
                Dl[m] = Contract<IO>::run(At, dh);
            }
        }

        if (grp == 3) {
#pragma unroll
            for (int m = 0; m < CPL; ++m) s_wl[bw][wv][n * CPL + m] = W[m][3];
        }
        if (lane == 63) s_c[bw][wv] = dk.c;
        __syncthreads();

        // ---- forward carriers (as in the forward kernel) ---------------------
        float ein[CPL], sin_[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { ein[m] = 0.f; sin_[m] = 0.f; }
        for (int r = 0; r < NW; ++r) {
            if (r % S == 0) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { e[m] = s[m]; s[m] = 0.f; }
            }
            if (r == wv) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { ein[m] = e[m]; sin_[m] = s[m]; }
            }
            const float c_ = s_c[bw][r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float wl = s_wl[bw][r][n * CPL + m];
                e[m] = c_ * e[m] + wl;
                s[m] = c_ * s[m] + wl;
            }
        }
        if (!out_step) continue;

        // ---- reverse carriers: from the end of the next step's first block --
        // back to this wave's sub-block.  eps is the full adjoint entering a
        // sub-block from the right, pr the one restarted at the block's end.
        float eps[CPL], pr[CPL], epsin[CPL], prin[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) { eps[m] = 0.f; pr[m] = 0.f; epsin[m] = 0.f; prin[m] = 0.f; }
        for (int r = S - 1; r >= 0; --r) {
            if (r % S == S - 1) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            const float c_ = s_cf[bn][r];
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float df = s_df[bn][r][n * CPL + m];
                eps[m] = c_ * eps[m] + df;
                pr[m] = c_ * pr[m] + df;
            }
        }
        for (int r = NW - 1; r >= wv; --r) {
            if (r % S == S - 1) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { eps[m] = pr[m]; pr[m] = 0.f; }
            }
            if (r == wv) {
#pragma unroll
                for (int m = 0; m < CPL; ++m) { epsin[m] = eps[m]; prin[m] = pr[m]; }
            } else {
                const float c_ = s_cf[bc][r];
#pragma unroll
                for (int m = 0; m < CPL; ++m) {
                    const float df = s_df[bc][r][n * CPL + m];
                    eps[m] = c_ * eps[m] + df;
                    pr[m] = c_ * pr[m] + df;
                }
            }
        }

        // ---- gradients ---------------------------------------------------------
        // r_q[k] = L[15][k] (last row of the sub-block operator) for this lane's rows.
        const int base = lane & 48;
        float R[4], Gsh[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) R[r] = shfl(dk.L[r], base + 15);
        // G[k-1] with G[-1] = 1: the decay product before each row.
        {
            const float gprev = shfl(dk.G[3], (lane - 16) & 63);   // G[4 grp - 1] from the row group above
            Gsh[0] = grp == 0 ? 1.0f : gprev;
            Gsh[1] = dk.G[0]; Gsh[2] = dk.G[1]; Gsh[3] = dk.G[2];
        }
        // Local state of the row above each of this lane's rows (0 above row 0).
        float wup[CPL];
#pragma unroll
        for (int m = 0; m < CPL; ++m) {
            const float v = shfl(W[m][3], (lane - 16) & 63);
            wup[m] = grp == 0 ? 0.0f : v;
        }
        float da_part[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t t = tr0 + r;
            float vdx[CPL], vdb[CPL], vdc[CPL];
            float acc = 0.f, acc2 = 0.f;
#pragma unroll
            for (int m = 0; m < CPL; ++m) {
                const float hv = W[m][r] + dk.G[r] * ein[m];           // jagged-window state
                const float dyv = dyr[r].get(m);
                vdc[m] = dyv * hv;
                const float du = Dl[m][r] + R[r] * epsin[m];           // adjoint of u
                const float dblk = Dl[m][r] + R[r] * prin[m];          // ... from this block's rows only
                vdx[m] = br[r].get(m) * du;
                if (p.residual) vdx[m] += dyv;
                vdb[m] = xr[r].get(m) * du;
                const float wprev = r == 0 ? wup[m] : W[m][r - 1];
                acc += wprev * du;
                acc2 += sin_[m] * du + (ein[m] - sin_[m]) * dblk;
            }
            da_part[r] = acc + Gsh[r] * acc2;
            if (t >= wk.t_begin && t < wk.t_end) {
                store_row<IO, CPL>(dxp + t * rs, vdx);
                store_row<IO, CPL>(dbp + t * rs, vdb);
                store_row<IO, CPL>(dcp + t * rs, vdc);
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float tot = row_sum(da_part[r]);
            const int64_t t = tr0 + r;
            if (n == 0 && t >= wk.t_begin && t < wk.t_end) dap[t * p.sa_t] = tot;
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
