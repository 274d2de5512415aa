// swr_api.cpp -- C ABI of the Sliding Window Recurrence library: argument
// validation (done entirely before any HIP runtime call), launch-shape
// selection and dispatch to the gfx950 kernels.
#include <stdint.h>

#include <algorithm>
#include <cstdlib>
#include <initializer_list>

#include "../../include/swr.h"
#include "swr_internal.h"
#include "swr_launch.h"

namespace {

constexpr int64_t kMaxWorkgroups = 0x7fffffffLL;
// Widest head: two virtual heads of 128 channels (one decay per head; their
// decay-gradient shares meet in two float32 atomic adds, which give the same
// sum in either order) or four of 64 (per-channel decay).
constexpr int64_t kMaxD = 256;
constexpr int64_t kMaxExtent = (int64_t)1 << 62;
// Default grid sizes, measured on the MI355X (256 compute units) over the
// benchmark workloads: the forward runs best with two 4-wave workgroups per
// CU; the backward with one 8-wave workgroup per CU, and with more, shorter
// runs when its workgroups are 4 waves (the lighter they are, the more).
// Longer runs mean fewer halo re-reads.
int64_t fwd_workgroups(const swr::Shape& s) { return s.tw * s.hw == 4 ? 512 : 256; }
int64_t bwd_workgroups(const swr::Shape& s, int cpl) {
    return s.tw * s.hw == 8 ? 256 : (cpl == 8 ? 1024 : 8192);
}

// Run length (tokens, a multiple of step) that splits each sequence into
// enough runs to give about `target` workgroups.
int64_t pick_run_len(int64_t T, int64_t seqs, int64_t step, int64_t target) {
    const int64_t nsteps = (T + step - 1) / step;
    const int64_t want = (target + seqs - 1) / seqs;
    const int64_t runs = std::max<int64_t>(1, std::min(nsteps, want));
    return ((nsteps + runs - 1) / runs) * step;
}

struct Dim {
    int64_t size, stride;
};

// Largest element offset of a strided tensor, or -1 on overflow / bad stride.
int64_t max_offset(const Dim* d, int nd) {
    int64_t off = 0;
    for (int i = 0; i < nd; ++i) {
        if (d[i].size <= 1) continue;
        if (d[i].stride < 0) return -1;
        if (d[i].stride > 0 && (d[i].size - 1) > kMaxExtent / d[i].stride) return -1;
        off += (d[i].size - 1) * d[i].stride;
        if (off > kMaxExtent) return -1;
    }
    return off;
}

// True when distinct index tuples never map to the same element.
bool non_overlapping(Dim* d, int nd) {
    std::sort(d, d + nd, [](const Dim& p, const Dim& q) { return p.stride < q.stride; });
    int64_t need = 1;   // smallest stride the next (larger-stride) dimension may have
    for (int i = 0; i < nd; ++i) {
        if (d[i].size <= 1) continue;
        if (d[i].stride < need) return false;
        need = d[i].stride * d[i].size;
    }
    return true;
}

struct Resolved {
    bool empty;
    int es;             // bytes per I/O element
    int cpl;            // channels per lane of the kernels = dk / 16
    bool pc;            // per-channel decay: a and da have the [B, T, H, D] layout of x
    int hshift;         // per-channel kernels: log2 of the virtual heads per head
    int pack;           // > 1: heads of 64 / pack channels packed into 64-channel virtual heads
    bool pair;          // forward: bf16 heads of 64 channels run two per kernel head (16-byte lane slices)
    int dk;             // channels a kernel's head covers (16, 32, 64 or 128)
    int dv;             // channels of a virtual head (D >> hshift), at most dk
    int nlane;          // lanes of a 16-lane row holding channels (dv / cpl)
    bool natural;       // D is 16, 32, 64 or 128, the widths every entry point accepts (the
                        // jagged window's forward, carriers and backward take any multiple of
                        // 16 up to kMaxD)
    int64_t hv;         // heads the kernels split the work over (H << hshift)
    int64_t vbytes;     // bytes of one lane's slice of an x-like row (alignment unit)
    swr::Shape bwd;     // backward workgroup shape
    swr::Shape fwd;     // forward workgroup shape
    int64_t step;       // a multiple of both sweeps' steps
    int64_t run_len, nruns, nwork;          // backward launch
    int64_t run_len_f, nruns_f, nwork_f;    // forward launch
    int64_t xspan;      // bytes spanned by one [B,T,H,D] tensor
    int64_t aspan;      // elements spanned by a / da
    int64_t nblocks;    // blocks per sequence
    int64_t carriers;   // float32 carriers of the whole problem
};

int resolve(const swr_problem_t* p, Resolved* r, bool allow_pack = true, bool allow_pair = false) {
    if (!p) return SWR_ERR_NULL;
    if (p->abi_version != SWR_ABI_VERSION) return SWR_ERR_VERSION;
    if (p->dtype != SWR_DTYPE_F32 && p->dtype != SWR_DTYPE_BF16) return SWR_ERR_DTYPE;
    if (p->B < 0 || p->T < 0 || p->H < 0 || p->D < 1) return SWR_ERR_SHAPE;
    if (p->block != 16 && p->block != 32 && p->block != 64 && p->block != 128) return SWR_ERR_BLOCK;
    if (p->D % 16 != 0 || p->D > kMaxD) return SWR_ERR_UNSUPPORTED;
    const uint32_t known = SWR_FLAG_RESIDUAL | SWR_FLAG_PER_CHANNEL_DECAY | SWR_FLAG_SIGMOID_DECAY |
                           SWR_FLAG_SIGMOID_PREGATE;
    if ((p->flags & ~known) != 0 || p->reserved != 0)
        return SWR_ERR_UNSUPPORTED;

    r->es = p->dtype == SWR_DTYPE_BF16 ? 2 : 4;
    r->pc = (p->flags & SWR_FLAG_PER_CHANNEL_DECAY) != 0;
    // A head wider than one kernel head is split into 2^hshift virtual heads
    // of dv channels; a virtual head narrower than the kernel's width dk (a
    // power of two) leaves the lanes past nlane idle.
    r->hshift = r->pc ? swr::pc_hshift(p->D) : swr::head_hshift(p->D);
    r->dv = (int)(p->D >> r->hshift);
    r->dk = r->dv <= 16 ? 16 : r->dv <= 32 ? 32 : r->dv <= 64 ? 64 : 128;
    r->natural = p->D == 16 || p->D == 32 || p->D == 64 || p->D == 128;
    r->pack = 1;
    // Heads of 16 or 32 channels stored next to each other run as packed
    // 64-channel virtual heads on the per-channel kernels (a lane slice of one
    // such head would be 2-4 bytes); the caller's pointers may still veto it
    // (alignment), see resolve_for.
    if (allow_pack && !r->pc && (p->D == 16 || p->D == 32) && p->H % (64 / p->D) == 0 && p->sx_h == p->D) {
        r->pack = (int)(64 / p->D);
        r->dk = 64;
    }
    // The jagged window's forward runs bf16 heads of 64 channels two at a
    // time, so that each lane moves 16-byte row slices as with 128-channel
    // heads and the tiles can be copied through LDS (the caller's pointers may
    // still veto it, see resolve_for).  The backward keeps them apart: two
    // heads' operators do not fit its register budget.
    // (Lane offsets then include the second head's share: sx_h of x and one
    // head's carriers, which must keep every 32-bit lane offset below 2^31
    // bytes.)
    const int64_t lim32 = 0x7fffffffLL;
    r->pair = allow_pair && !r->pc && p->D == 64 && p->dtype == SWR_DTYPE_BF16 && p->H % 2 == 0 &&
              (p->sx_h * 2) % 16 == 0 && p->sx_h >= 0 && p->sx_h <= (int64_t)1 << 26 && p->sa_h >= 0 &&
              p->sa_h <= (int64_t)1 << 26 && p->sx_t >= 0 && p->sx_t <= (lim32 - p->sx_h * 2 - 128) / 32 &&
              p->sa_t >= 0 && p->sa_t <= (lim32 - p->sa_h * 4) / 64 &&
              (p->T + p->block - 1) / p->block <= lim32 / (2 * 64 * 4);
    if (r->pair) r->dk = 128;
    r->cpl = r->dk / 16;
    r->nlane = r->pack > 1 || r->pair ? 16 : r->dv / r->cpl;
    r->hv = r->pack > 1 ? p->H / r->pack : r->pair ? p->H / 2 : p->H << r->hshift;
    r->vbytes = std::min<int64_t>(16, (int64_t)(r->dk / 16) * r->es);
    r->bwd = swr::bwd_shape(p->block, r->hv);
    r->fwd = swr::fwd_shape(p->block, r->hv);
    r->step = (int64_t)std::max(r->bwd.tw, r->fwd.tw) * 16;   // both sweeps' steps divide a run
    if (p->run_len < 0 || (p->run_len > 0 && p->run_len % r->step != 0)) return SWR_ERR_UNSUPPORTED;

    r->empty = p->B == 0 || p->T == 0 || p->H == 0;
    r->xspan = r->aspan = 0;
    if (!r->empty) {   // strides of an empty tensor are meaningless
        Dim xd[4] = {{p->B, p->sx_b}, {p->T, p->sx_t}, {p->H, p->sx_h}, {p->D, 1}};
        const int64_t xo = max_offset(xd, 4);
        if (xo < 0 || !non_overlapping(xd, 4)) return SWR_ERR_SHAPE;
        r->xspan = (xo + 1) * r->es;
        if (r->pc) {       // a and da use the strides of x; sa_* are not read
            r->aspan = xo + 1;
        } else {
            Dim ad[3] = {{p->B, p->sa_b}, {p->T, p->sa_t}, {p->H, p->sa_h}};
            const int64_t ao = max_offset(ad, 3);
            if (ao < 0 || !non_overlapping(ad, 3)) return SWR_ERR_SHAPE;
            r->aspan = ao + 1;
        }
    }
    const int64_t seqs = p->B * r->hv;             // (batch, head) sequences the kernels see
    if (r->fwd.hw > 1 && p->run_len == 0 && !r->empty) {
        // On a problem too small to fill the forward's grid, grouping heads
        // would only halve it: keep one head per workgroup there.
        const int64_t g = seqs / r->fwd.hw;
        const int64_t rl = pick_run_len(p->T, g, r->step, fwd_workgroups(r->fwd));
        if (g * ((p->T + rl - 1) / rl) < fwd_workgroups(r->fwd)) r->fwd = swr::fwd_shape_single();
    }
    const int64_t groups = seqs / r->fwd.hw;       // forward work items per run position
    const int64_t groups_b = seqs / r->bwd.hw;     // backward work items per run position
    if (p->run_len > 0) {
        r->run_len = r->run_len_f = p->run_len;
    } else if (r->empty) {
        r->run_len = r->run_len_f = r->step;
    } else {
        r->run_len = pick_run_len(p->T, groups_b, r->step, bwd_workgroups(r->bwd, r->cpl));
        r->run_len_f = pick_run_len(p->T, groups, r->step, fwd_workgroups(r->fwd));
    }
    r->nruns = r->empty ? 0 : (p->T + r->run_len - 1) / r->run_len;
    r->nruns_f = r->empty ? 0 : (p->T + r->run_len_f - 1) / r->run_len_f;
    if (!r->empty && std::max(r->nruns, r->nruns_f) > kMaxWorkgroups / seqs) return SWR_ERR_UNSUPPORTED;
    r->nwork = groups_b * r->nruns;
    r->nwork_f = groups * r->nruns_f;
    r->nblocks = (p->T + p->block - 1) / p->block;
    r->carriers = p->B * p->H * r->nblocks * p->D;
    if (!r->empty) {
        // The kernels address a lane's data with 32-bit byte offsets from a
        // per-step base: 16 rows of x-like tensors, 16 tokens of a / da, and a
        // (batch, head)'s carrier array must stay below 2^31 bytes.
        const int64_t lim = 0x7fffffffLL;
        if (p->sx_t > (lim - p->D * r->es) / (16 * r->es)) return SWR_ERR_UNSUPPORTED;
        if (r->pc ? p->sx_t > (lim - p->D * 4) / (16 * 4) : p->sa_t > lim / (16 * 4))
            return SWR_ERR_UNSUPPORTED;
        if (r->nblocks > lim / (p->D * 4)) return SWR_ERR_UNSUPPORTED;
    }
    return SWR_OK;
}

int check_strides_aligned(const swr_problem_t* p, const Resolved& r) {
    const int64_t vda = std::min<int64_t>(16, (int64_t)(r.dk / 16) * 4);   // per-channel da slice
    const Dim xd[3] = {{p->B, p->sx_b}, {p->T, p->sx_t}, {p->H, p->sx_h}};
    for (const Dim& d : xd) {
        if (d.size > 1 && (d.stride * r.es) % r.vbytes != 0) return SWR_ERR_ALIGN;
        if (r.pc && d.size > 1 && (d.stride * 4) % vda != 0) return SWR_ERR_ALIGN;
    }
    if ((r.pc || r.hshift) && (r.dv * r.es) % r.vbytes != 0) return SWR_ERR_ALIGN;   // a virtual head's offset
    return SWR_OK;
}

bool aligned(const void* ptr, int64_t bytes) { return ((uintptr_t)ptr % (uintptr_t)bytes) == 0; }

// resolve() for a call with these [B,T,H,D] tensors: packed small heads need
// each lane's 64-channel row slice aligned (8 or 16 bytes); otherwise the
// heads run one by one.
// The same for paired 64-channel heads (allow_pair: the jagged window's
// forward and backward), which need 16-byte aligned slices.
int resolve_for(const swr_problem_t* p, Resolved* r, std::initializer_list<const void*> xs,
                bool allow_pair = false) {
    int rc = resolve(p, r, true, allow_pair);
    if (rc != SWR_OK || (r->pack == 1 && !r->pair) || r->empty) return rc;
    bool ok = check_strides_aligned(p, *r) == SWR_OK;
    for (const void* q : xs)
        if (q && !aligned(q, r->vbytes)) ok = false;
    return ok ? SWR_OK : resolve(p, r, false, false);
}

struct Span {
    uintptr_t lo, hi;   // [lo, hi)
};

Span span(const void* p, int64_t bytes) { return {(uintptr_t)p, (uintptr_t)p + (uintptr_t)bytes}; }

bool overlap(const Span& a, const Span& b) { return a.lo < b.hi && b.lo < a.hi; }

// Polls a chunk of the one-pass exact recurrence makes before it gives up
// waiting for an earlier chunk's publication: 2^16, unless the environment
// variable SWR_CHAIN_SPIN_LIMIT (read at every call) lowers it, so that tests
// can force the time-out path; it can never raise it.
int32_t chain_spin_limit() {
    constexpr long kDefault = 1L << 16;
    const char* s = std::getenv("SWR_CHAIN_SPIN_LIMIT");
    if (s && *s) {
        char* end = nullptr;
        const long v = std::strtol(s, &end, 10);
        if (*end == '\0' && v >= 0 && v < kDefault) return (int32_t)v;
    }
    return (int32_t)kDefault;
}

swr::Params make_params(const swr_problem_t* p, const Resolved& r, bool backward) {
    swr::Params k{};
    k.B = p->B; k.T = p->T; k.H = p->H;
    k.Hv = r.hv;
    k.hshift = r.hshift;
    k.dh = (int32_t)p->D;
    k.dv = r.pack > 1 ? 64 : r.pair ? 128 : r.dv;
    k.nlane = r.nlane;
    k.sx_b = p->sx_b; k.sx_t = p->sx_t; k.sx_h = p->sx_h;
    k.sa_b = p->sa_b; k.sa_t = p->sa_t; k.sa_h = p->sa_h;
    k.block = (int32_t)p->block;
    k.lshift = p->block == 16 ? 4 : p->block == 32 ? 5 : p->block == 64 ? 6 : 7;
    k.residual = (p->flags & SWR_FLAG_RESIDUAL) ? 1 : 0;
    k.sig_a = (p->flags & SWR_FLAG_SIGMOID_DECAY) ? 1 : 0;
    k.sig_b = (p->flags & SWR_FLAG_SIGMOID_PREGATE) ? 1 : 0;
    k.run_len = backward ? r.run_len : r.run_len_f;
    k.nruns = backward ? r.nruns : r.nruns_f;
    k.nwork = backward ? r.nwork : r.nwork_f;
    k.nblocks = r.nblocks;
    k.spin_limit = chain_spin_limit();
    return k;
}

}  // namespace

extern "C" {

int swr_abi_version(void) { return SWR_ABI_VERSION; }

const char* swr_error_string(int code) {
    switch (code) {
        case SWR_OK: return "success";
        case SWR_ERR_NULL: return "a required pointer is NULL";
        case SWR_ERR_SHAPE: return "invalid shape or strides (negative size, D < 1, overlapping or overflowing strides)";
        case SWR_ERR_DTYPE: return "unknown dtype";
        case SWR_ERR_BLOCK: return "block must be 16, 32, 64 or 128";
        case SWR_ERR_ALIGN: return "pointer or stride not aligned to the per-lane vector width";
        case SWR_ERR_ALIAS: return "an output overlaps an input or another output";
        case SWR_ERR_UNSUPPORTED: return "unsupported: D must be a multiple of 16 up to 256 (16, 32, 64 or 128 except for swr_forward, swr_carriers and swr_backward); unknown flags; bad run_len; or offsets beyond 32 bits";
        case SWR_ERR_HIP: return "the HIP runtime rejected the kernel launch";
        case SWR_ERR_VERSION: return "ABI version mismatch";
        case SWR_ERR_SCRATCH: return "the problem needs more workspace than the library's static scratch array holds (SWR_NOALLOC_SCRATCH_BYTES)";
        default: return "unknown status code";
    }
}

int swr_launch_info(const swr_problem_t* problem, int64_t* fwd_run_len, int64_t* fwd_workgroups,
                    int64_t* bwd_run_len, int64_t* bwd_workgroups) {
    // the plans of swr_forward (which may pair heads) and swr_backward, with
    // suitably aligned pointers
    Resolved r, f;
    int rc = resolve(problem, &r);
    if (rc != SWR_OK) return rc;
    if ((rc = resolve(problem, &f, true, true)) != SWR_OK) return rc;
    if (fwd_run_len) *fwd_run_len = f.run_len_f;
    if (fwd_workgroups) *fwd_workgroups = f.nwork_f;
    if (bwd_run_len) *bwd_run_len = r.run_len;
    if (bwd_workgroups) *bwd_workgroups = r.nwork;
    return SWR_OK;
}

int64_t swr_carrier_elems(const swr_problem_t* problem) {
    Resolved r;
    const int rc = resolve(problem, &r);
    return rc != SWR_OK ? rc : r.carriers;
}

namespace {

// Shared by swr_forward (y != NULL) and swr_carriers (y == NULL).
int forward_impl(const swr_problem_t* p, const void* x, const void* a, const void* b,
                 const void* c, void* y, float* carriers, void* stream) {
    Resolved r;
    int rc = resolve_for(p, &r, {x, b, c, (const void*)y}, true);
    if (rc != SWR_OK) return rc;
    if (r.empty) return SWR_OK;
    if (!x || !a || !b || (y && !c)) return SWR_ERR_NULL;
    for (const void* q : {x, b, c, (const void*)y})
        if (q && !aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
    if (!aligned(a, r.pc ? r.vbytes : r.es) || (carriers && !aligned(carriers, 16))) return SWR_ERR_ALIGN;
    if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    const Span ins[4] = {span(x, r.xspan), span(b, r.xspan), span(c, c ? r.xspan : 0),
                         span(a, r.aspan * r.es)};
    const Span sy = span(y, y ? r.xspan : 0), sv = span(carriers, carriers ? r.carriers * 4 : 0);
    for (const Span& s : ins)
        if (overlap(sy, s) || overlap(sv, s)) return SWR_ERR_ALIAS;
    if (overlap(sy, sv)) return SWR_ERR_ALIAS;

    swr::Params k = make_params(p, r, false);
    k.x = x; k.a = a; k.b = b; k.c = c; k.y = y; k.carriers = carriers;
    return swr::launch(k, p->dtype, r.dk, r.fwd, false, r.pc, r.pack, r.pair ? swr::kPaired : swr::kSwr,
                       stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

}  // namespace

int swr_forward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                const void* c, void* y, float* carriers, void* stream) {
    Resolved r;
    const int rc = resolve(p, &r);
    if (rc != SWR_OK) return rc;
    if (!r.empty && !y) return SWR_ERR_NULL;
    return forward_impl(p, x, a, b, c, y, carriers, stream);
}

int swr_carriers(const swr_problem_t* p, const void* x, const void* a, const void* b,
                 float* carriers, void* stream) {
    Resolved r;
    const int rc = resolve(p, &r);
    if (rc != SWR_OK) return rc;
    if (!r.empty && !carriers) return SWR_ERR_NULL;
    return forward_impl(p, x, a, b, nullptr, nullptr, carriers, stream);
}

int swr_backward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                 const void* c, const void* dy, const float* carriers, void* dx, float* da,
                 void* db, void* dc, void* stream) {
    Resolved r;
    int rc = resolve_for(p, &r, {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc});
    if (rc != SWR_OK) return rc;
    if (r.empty) return SWR_OK;
    // (carriers may be NULL: the kernels then recompute them)
    if (!x || !a || !b || !c || !dy || !dx || !da || !db || !dc) return SWR_ERR_NULL;
    for (const void* q : {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc})
        if (!aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
    const int64_t va = r.pc ? r.vbytes : r.es;
    const int64_t vda = r.pc ? std::min<int64_t>(16, (int64_t)(r.dk / 16) * 4) : 4;
    if (!aligned(a, va) || !aligned(da, vda) || (carriers && !aligned(carriers, 16))) return SWR_ERR_ALIGN;
    if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    const Span outs[4] = {span(dx, r.xspan), span(db, r.xspan), span(dc, r.xspan),
                          span(da, r.aspan * 4)};
    const Span ins[6] = {span(x, r.xspan), span(b, r.xspan), span(c, r.xspan), span(dy, r.xspan),
                         span(a, r.aspan * r.es), span(carriers, carriers ? r.carriers * 4 : 0)};
    for (int i = 0; i < 4; ++i) {
        for (const Span& s : ins)
            if (overlap(outs[i], s)) return SWR_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], outs[j])) return SWR_ERR_ALIAS;
    }

    swr::Params k = make_params(p, r, true);
    k.x = x; k.a = a; k.b = b; k.c = c; k.dy = dy;
    k.dx = dx; k.da = da; k.db = db; k.dc = dc;
    k.carriers = const_cast<float*>(carriers);
    return swr::launch(k, p->dtype, r.dk, r.bwd, true, r.pc, r.pack, carriers ? swr::kSwr : swr::kRecompute,
                       stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Exact (untruncated) recurrence
// ---------------------------------------------------------------------------

namespace {

// The backward's stage I reads only c, dy and a and has no block structure:
// it runs 4-wave groups over runs finer than the backward's own (halving
// them while fewer than ~2048 groups would result), so that it streams at
// the rate of a read-only pass.  Returns the aggregate run length (a
// divisor of the backward's run length, a multiple of 64 tokens).
int64_t bwd_agg_len(const swr_problem_t* p, const Resolved& r) {
    const int64_t seqs = p->B * r.hv;
    int64_t len = r.run_len;
    while (len % 128 == 0 && seqs * ((p->T + len - 1) / len) < 2048) len /= 2;
    return len;
}

// Workspace of the exact recurrence, in float32 elements: per (batch, head)
// and aggregate run, the run's aggregate end state (D), the value entering
// the run (D) and the run's decay product (1, or D for a per-channel decay),
// for the largest of the launches' run counts.
struct ExactWs {
    int64_t nr;       // runs per sequence the workspace is laid out for
    int64_t floats;   // total float32 elements
};

ExactWs exact_ws(const swr_problem_t* p, const Resolved& r) {
    ExactWs w;
    const int64_t na = r.empty ? 0 : (p->T + bwd_agg_len(p, r) - 1) / bwd_agg_len(p, r);
    w.nr = std::max(std::max(r.nruns, r.nruns_f), na);
    // a per-channel decay has one run decay product per channel
    w.floats = p->B * p->H * w.nr * (2 * p->D + (r.pc || r.pack > 1 ? p->D : 1));
    return w;
}



// The exact forward in one pass (swr_chain.hip).  With one decay per head
// on the MFMA kernels a float32 head of 128 channels runs as two virtual
// heads of 64, each its own chain of chunks: the lighter wave lets two
// workgroups share a compute unit, which hides the look-back's latency; a
// bf16 head of 128 stays whole (16-byte row slices a lane; the kernel keeps
// its local solutions in LDS to fit two workgroups a compute unit).
// Workspace: two ticket counters (padded to 16 floats), then per chunk of
// chain_tokens() tokens of every virtual sequence a flag and a decay product,
// then per chunk an aggregate end state and an inclusive end state (a
// virtual head's channels each).  With a decay per channel the per-channel
// kernels' virtual heads chain the same way with a decay product per channel:
// the flags (padded to 4), then a decay product, an aggregate and an
// inclusive state per chunk and channel.
#ifndef SWR_EXACT_CHAIN
#define SWR_EXACT_CHAIN 1
#endif

struct ChainWs {
    int cpl;          // channels per lane of the launch
    int hs;           // log2 of the virtual heads per head (shared decay)
    bool pcp;         // decay products per channel (a decay per channel)
    int64_t nch;      // chunks per sequence
    int64_t n;        // chunks of the (virtual) sequences
    int64_t dv;       // channels of a (virtual) sequence
    int64_t floats;   // float32 elements
};

ChainWs chain_ws(const swr_problem_t* p, const Resolved& r) {
    ChainWs c;
    const int64_t ct = swr::chain_tokens();
    c.nch = (p->T + ct - 1) / ct;
    c.pcp = r.pc;
    if (c.pcp) {   // the per-channel kernels' virtual heads; a flag, then three values a channel
        c.cpl = r.cpl;
        c.hs = 0;
        c.dv = 16 * r.cpl;
        c.n = p->B * r.hv * c.nch;
        c.floats = 16 + (c.n + 3) / 4 * 4 + 3 * c.n * c.dv;
        return c;
    }
    c.cpl = (int)std::min<int64_t>(p->D / 16, p->dtype == 1 ? 8 : 4);
    c.hs = 0;
    while ((16 * c.cpl) << c.hs < p->D) ++c.hs;
    c.dv = 16 * c.cpl;
    c.n = (p->B * p->H << c.hs) * c.nch;
    // ticket counters, a flag and a decay product per chunk, two D-vectors per real chunk
    c.floats = 16 + 2 * c.n + 2 * (c.n >> c.hs) * p->D;
    return c;
}

// The tickets are 32-bit counters (each workgroup takes one past the last chunk).
// Packed small heads keep the three stages: at B8 T16384 H16 d16 (32 packed
// sequences of 128 chunks) the chain's boundaries, not the bytes, set the
// time (99 against 94 us).
bool use_chain(const swr_problem_t* p, const Resolved& r) {
    return SWR_EXACT_CHAIN && !r.empty && r.pack == 1 && chain_ws(p, r).n < ((int64_t)1 << 30);
}

// The backward in one pass, for heads of up to 64 channels, where it
// measured faster than the three stages (B1 T131072 H32 d64: 1047 -> 928 us;
// B16 T8192 H32 d64: 960 -> 895 us); with 128 channels it is slower (983 ->
// 1208 us: one workgroup a compute unit, whose look-back nothing covers).
#ifndef SWR_EXACT_CHAIN_BWD
#define SWR_EXACT_CHAIN_BWD 1
#endif
bool use_chain_bwd(const swr_problem_t* p, const Resolved& r) {
    if (!SWR_EXACT_CHAIN_BWD || !use_chain(p, r)) return false;
    const ChainWs cw = chain_ws(p, r);
    return !cw.pcp && cw.hs == 0 && cw.cpl <= 4;
}

// The one-pass forward of bf16 heads of 64 channels taken two at a time
// (16-byte lane slices): the per-channel layout over the pairs' 128 channels.
int64_t chain_pair_floats(const swr_problem_t* p) {
    const int64_t ct = swr::chain_tokens();
    const int64_t n = p->B * (p->H / 2) * ((p->T + ct - 1) / ct);
    return 16 + (n + 3) / 4 * 4 + 3 * n * 128;
}
// Whether the problem's shape and strides let heads run in pairs (the
// pointers are checked where there are any: resolve_for).
bool shape_pairs(const swr_problem_t* p) {
    Resolved t;
    return resolve(p, &t, true, true) == SWR_OK && t.pair && !t.empty && t.hv < ((int64_t)1 << 30);
}

// Workspace of the exact calls for one plan: the three-stage arrays (the
// backward's, and the forward's when it does not run in one pass) or the
// one-pass forward's, whichever is larger.
int64_t exact_ws_floats(const swr_problem_t* p, const Resolved& r) {
    int64_t f = std::max(exact_ws(p, r).floats, use_chain(p, r) ? chain_ws(p, r).floats : (int64_t)0);
    if (use_chain(p, r) && !r.pc && shape_pairs(p)) f = std::max(f, chain_pair_floats(p));
    return f;
}

// Pointers into the workspace for one launch.
void exact_arrays(const swr_problem_t* p, const ExactWs& w, void* ws, float** v, float** carry, float** prod) {
    float* f = (float*)ws;
    const int64_t n = p->B * p->H * w.nr * p->D;
    *v = f;
    *carry = f + n;
    *prod = f + 2 * n;
}

}  // namespace

extern "C" {

int64_t swr_exact_workspace_bytes(const swr_problem_t* problem) {
    // enough for either launch plan (packed small heads or not), since the
    // pointers of the later call decide between them
    Resolved r, u;
    int rc = resolve(problem, &r, true);
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    if ((rc = resolve(problem, &u, false)) != SWR_OK) return rc;
    return std::max(exact_ws_floats(problem, r), exact_ws_floats(problem, u)) * 4;
}

int swr_exact_forward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                      const void* c, const float* h0, void* y, float* carriers, float* h_last,
                      void* workspace, void* stream) {
    return swr::exact_forward_impl(p, x, a, b, c, h0, y, carriers, h_last, workspace, nullptr, 0, stream);
}

}  // extern "C"

int swr::exact_forward_impl(const swr_problem_t* p, const void* x, const void* a, const void* b,
                            const void* c, const float* h0, void* y, float* carriers, float* h_last,
                            void* workspace, ScratchFn scratch, int64_t scratch_bytes, void* stream) {
    Resolved r;
    int rc = resolve_for(p, &r, {x, b, c, (const void*)y});
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    const ExactWs w = exact_ws(p, r);
    // the library's static array may hold the three stages' arrays but not the
    // one pass's: the allocation-free call then runs the three stages.  bf16
    // heads of 64 channels run in pairs where the pointers and strides allow.
#ifndef SWR_EXACT_CHAIN_PAIR
#define SWR_EXACT_CHAIN_PAIR 1
#endif
    Resolved rp;
    const bool pair = SWR_EXACT_CHAIN_PAIR && use_chain(p, r) && !r.pc && resolve_for(p, &rp, {x, b, c, (const void*)y}, true) == SWR_OK &&
                      rp.pair && (!scratch || chain_pair_floats(p) * 4 <= scratch_bytes);
    const bool chain = !pair && use_chain(p, r) && (!scratch || chain_ws(p, r).floats * 4 <= scratch_bytes);
    const int64_t wfloats = pair ? chain_pair_floats(p) : chain ? chain_ws(p, r).floats : w.floats;
    const int64_t seqs = p->B * p->H, sbytes = seqs * p->D * 4;
    if (seqs == 0) return SWR_OK;
    if (!r.empty && (!x || !a || !b || !c || !y)) return SWR_ERR_NULL;
    if (scratch) {
        // the library's own array: disjoint from every caller buffer, located later
        if (wfloats * 4 > scratch_bytes) return SWR_ERR_SCRATCH;
        workspace = nullptr;
    } else if (wfloats > 0 && !workspace) {
        return SWR_ERR_NULL;
    }
    for (const void* q : {(const void*)h0, (const void*)h_last, (const void*)carriers, (const void*)workspace})
        if (q && !aligned(q, 16)) return SWR_ERR_ALIGN;
    if (!r.empty) {
        for (const void* q : {x, b, c, (const void*)y})
            if (!aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
        if (!aligned(a, r.pc ? r.vbytes : r.es)) return SWR_ERR_ALIGN;
        if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    }
    const Span ins[5] = {span(x, r.xspan), span(b, r.xspan), span(c, r.xspan), span(a, r.aspan * r.es),
                         span(h0, h0 ? sbytes : 0)};
    const Span outs[4] = {span(y, r.xspan), span(carriers, carriers ? r.carriers * 4 : 0),
                          span(h_last, h_last ? sbytes : 0), span(workspace, workspace ? wfloats * 4 : 0)};
    for (int i = 0; i < 4; ++i) {
        for (const Span& s : ins)
            if (overlap(outs[i], s)) return SWR_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], outs[j])) return SWR_ERR_ALIAS;
    }

    if (scratch && wfloats > 0 && !(workspace = scratch(stream))) return SWR_ERR_HIP;
    if (pair) {   // one pass, heads of 64 channels two at a time
        const int64_t nch = (p->T + swr::chain_tokens() - 1) / swr::chain_tokens();
        const int64_t n = p->B * (p->H / 2) * nch;
        float* f = (float*)workspace;
        swr::Params k = make_params(p, r, false);
        k.x = x; k.a = a; k.b = b; k.c = c; k.y = y; k.carriers = carriers; k.h0 = h0; k.h_last = h_last;
        k.chain_ctr = (int32_t*)f;
        k.chain_flags = (int32_t*)(f + 16);
        k.agg_p = f + 16 + (n + 3) / 4 * 4;
        k.agg_v = k.agg_p + n * 128;
        k.chain_incl = k.agg_v + n * 128;
        k.nruns = nch;
        k.nwork = std::min<int64_t>(n, 512);   // two workgroups a compute unit
        return swr::launch_chain_forward_pair(k, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
    }
    if (chain && chain_ws(p, r).pcp) {   // one pass, a decay per channel
        const ChainWs cw = chain_ws(p, r);
        float* f = (float*)workspace;
        swr::Params k = make_params(p, r, false);
        k.x = x; k.a = a; k.b = b; k.c = c; k.y = y; k.carriers = carriers; k.h0 = h0; k.h_last = h_last;
        k.chain_ctr = (int32_t*)f;
        k.chain_flags = (int32_t*)(f + 16);
        k.agg_p = f + 16 + (cw.n + 3) / 4 * 4;
        k.agg_v = k.agg_p + cw.n * cw.dv;
        k.chain_incl = k.agg_v + cw.n * cw.dv;
        k.nruns = cw.nch;
        // persistent workgroups: as many as the 256 compute units hold at once
        k.nwork = std::min<int64_t>(cw.n, 256 * (cw.cpl == 1 ? 3 : 2));
        return swr::launch_chain_forward_pc(k, p->dtype, cw.cpl, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
    }
    if (chain) {   // one pass: chained chunks with a look-back
        const ChainWs cw = chain_ws(p, r);
        float* f = (float*)workspace;
        swr::Params k = make_params(p, r, false);
        k.x = x; k.a = a; k.b = b; k.c = c; k.y = y; k.carriers = carriers; k.h0 = h0; k.h_last = h_last;
        k.chain_ctr = (int32_t*)f;
        k.chain_flags = (int32_t*)(f + 16);
        k.agg_p = f + 16 + cw.n;
        k.agg_v = f + 16 + 2 * cw.n;
        k.chain_incl = k.agg_v + (cw.n >> cw.hs) * p->D;
        k.hshift = cw.hs;
        k.Hv = p->H << cw.hs;
        k.dh = (int32_t)p->D;
        k.dv = (int32_t)(16 * cw.cpl);
        k.nruns = cw.nch;
        // persistent workgroups: as many as the 256 compute units hold at once
        // (registers: bf16 with 16 or 8 channels a lane 2 or 3, float32 with
        // 8 channels 2, 2 and 1 channels 2 and 3)
        const bool bf16 = p->dtype == 1;
        const int per_cu = cw.cpl == 8 ? 2 : cw.cpl == 4 ? (bf16 ? 3 : 2) : cw.cpl == 1 ? 3 : 2;
        k.nwork = std::min<int64_t>(cw.n, 256 * per_cu);
        return swr::launch_chain_forward(k, p->dtype, cw.cpl, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
    }
    float *wv = nullptr, *wc = nullptr, *wp = nullptr;
    if (w.floats > 0) exact_arrays(p, w, workspace, &wv, &wc, &wp);
    swr::Params k = make_params(p, r, false);
    k.x = x; k.a = a; k.b = b; k.c = c;
    k.agg_v = wv; k.agg_p = wp; k.carry = wc;
    k.agg_len = k.run_len; k.agg_nruns = k.nruns;
    // Stage I: local solves of every run, keeping each run's end state and decay product.
    if (!r.empty && swr::launch(k, p->dtype, r.dk, r.fwd, false, r.pc, r.pack, swr::kAggregate, stream) != hipSuccess)
        return SWR_ERR_HIP;
    // Stage II: the carrier recurrence over the runs, from h0; h_last is its final value.
    swr::ScanParams q{};
    q.agg_v = wv; q.agg_p = wp; q.carry = wc; q.init = h0; q.fin = h_last;
    q.seqs = seqs; q.nruns = r.empty ? 0 : k.nruns; q.D = (int32_t)p->D; q.reverse = 0;
    q.p_per_channel = r.pc || r.pack > 1 ? 1 : 0;
    if ((h_last || !r.empty) && swr::launch_scan(q, stream) != hipSuccess) return SWR_ERR_HIP;
    if (r.empty) return SWR_OK;
    // Stage III: every run again from its exact entering state: outputs and exact block carriers.
    k.y = y; k.carriers = carriers;
    return swr::launch(k, p->dtype, r.dk, r.fwd, false, r.pc, r.pack, swr::kExact, stream) == hipSuccess ? SWR_OK
                                                                                          : SWR_ERR_HIP;
}

extern "C" {

int swr_exact_backward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                       const void* c, const void* dy, const float* h0, const float* carriers,
                       const float* dh_last, void* dx, float* da, void* db, void* dc, float* dh0,
                       void* workspace, void* stream) {
    Resolved r;
    int rc = resolve_for(p, &r, {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc});
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    const ExactWs w = exact_ws(p, r);
    const int64_t wfloats = exact_ws_floats(p, r);
    const int64_t seqs = p->B * p->H, sbytes = seqs * p->D * 4;
    if (seqs == 0) return SWR_OK;
    if (!r.empty && (!x || !a || !b || !c || !dy || !carriers || !dx || !da || !db || !dc)) return SWR_ERR_NULL;
    if (wfloats > 0 && !workspace) return SWR_ERR_NULL;
    for (const void* q : {(const void*)h0, (const void*)dh_last, (const void*)dh0, (const void*)carriers,
                          (const void*)workspace})
        if (q && !aligned(q, 16)) return SWR_ERR_ALIGN;
    if (!r.empty) {
        for (const void* q : {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc})
            if (!aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
        const int64_t vda = r.pc ? std::min<int64_t>(16, (int64_t)(r.dk / 16) * 4) : 4;
        if (!aligned(a, r.pc ? r.vbytes : r.es) || !aligned(da, vda)) return SWR_ERR_ALIGN;
        if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    }
    const Span ins[8] = {span(x, r.xspan), span(b, r.xspan), span(c, r.xspan), span(dy, r.xspan),
                         span(a, r.aspan * r.es), span(carriers, carriers ? r.carriers * 4 : 0),
                         span(h0, h0 ? sbytes : 0), span(dh_last, dh_last ? sbytes : 0)};
    const Span outs[6] = {span(dx, r.xspan), span(db, r.xspan), span(dc, r.xspan), span(da, r.aspan * 4),
                          span(dh0, dh0 ? sbytes : 0), span(workspace, wfloats * 4)};
    for (int i = 0; i < 6; ++i) {
        for (const Span& s : ins)
            if (overlap(outs[i], s)) return SWR_ERR_ALIAS;
        for (int j = i + 1; j < 6; ++j)
            if (overlap(outs[i], outs[j])) return SWR_ERR_ALIAS;
    }

    if (use_chain_bwd(p, r)) {   // one pass: chunks from the sequences' ends, chained by a look-back
        const ChainWs cw = chain_ws(p, r);
        float* f = (float*)workspace;
        swr::Params k = make_params(p, r, true);
        k.x = x; k.a = a; k.b = b; k.c = c; k.dy = dy;
        k.dx = dx; k.da = da; k.db = db; k.dc = dc;
        k.carriers = const_cast<float*>(carriers); k.h0 = h0; k.dh_last = dh_last; k.dh0 = dh0;
        k.chain_ctr = (int32_t*)f;
        k.chain_flags = (int32_t*)(f + 16);
        k.agg_p = f + 16 + cw.n;
        k.agg_v = f + 16 + 2 * cw.n;
        k.chain_incl = k.agg_v + cw.n * p->D;
        k.nruns = cw.nch;
        // persistent workgroups: as many as the 256 compute units hold at once
        k.nwork = std::min<int64_t>(cw.n, 256 * (cw.cpl == 8 ? 1 : 2));
        return swr::launch_chain_backward(k, p->dtype, cw.cpl, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
    }
    float *wv = nullptr, *wc = nullptr, *wp = nullptr;
    if (w.floats > 0) exact_arrays(p, w, workspace, &wv, &wc, &wp);
    swr::Params k = make_params(p, r, true);
    k.x = x; k.a = a; k.b = b; k.c = c; k.dy = dy;
    k.agg_v = wv; k.agg_p = wp; k.carry = wc; k.h0 = h0;
    k.agg_len = r.empty ? 1 : bwd_agg_len(p, r);
    k.agg_nruns = r.empty ? 0 : (p->T + k.agg_len - 1) / k.agg_len;
    // Stage I: reverse local solves of every aggregate run (from c, dy, a), 4-wave groups.
    if (!r.empty) {
        swr::Params ka = k;
        ka.run_len = k.agg_len;
        ka.nruns = k.agg_nruns;
        ka.nwork = p->B * r.hv * k.agg_nruns;
        if (swr::launch(ka, p->dtype, r.dk, swr::Shape{4, 1}, true, r.pc, r.pack, swr::kAggregate, stream) !=
            hipSuccess)
            return SWR_ERR_HIP;
    }
    // Stage II: the reverse carrier recurrence over the aggregate runs, from dh_last; dh0 is
    // its final value.
    swr::ScanParams q{};
    q.agg_v = wv; q.agg_p = wp; q.carry = wc; q.init = dh_last; q.fin = dh0;
    q.seqs = seqs; q.nruns = k.agg_nruns; q.D = (int32_t)p->D; q.reverse = 1;
    q.p_per_channel = r.pc || r.pack > 1 ? 1 : 0;
    if ((dh0 || !r.empty) && swr::launch_scan(q, stream) != hipSuccess) return SWR_ERR_HIP;
    if (r.empty) return SWR_OK;
    // Stage III: the gradients, from the adjoint entering each run and the exact block carriers.
    k.dx = dx; k.da = da; k.db = db; k.dc = dc;
    k.carriers = const_cast<float*>(carriers);
    return swr::launch(k, p->dtype, r.dk, r.bwd, true, r.pc, r.pack, swr::kExact, stream) == hipSuccess ? SWR_OK
                                                                                         : SWR_ERR_HIP;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Recurrent steps and the decoding state
// ---------------------------------------------------------------------------

namespace {

// Bytes of one thread's slice of a row in the step and state kernels: D/16
// channels (the whole head is one slice set even for a per-channel decay).
int64_t step_vbytes(const swr_problem_t* p, const Resolved& r) {
    return std::min<int64_t>(16, (p->D / 16) * r.es);
}

int check_step_strides(const swr_problem_t* p, const Resolved& r, int64_t vb) {
    const Dim xd[3] = {{p->B, p->sx_b}, {p->T, p->sx_t}, {p->H, p->sx_h}};
    for (const Dim& d : xd)
        if (d.size > 1 && (d.stride * r.es) % vb != 0) return SWR_ERR_ALIGN;
    return SWR_OK;
}

int step_impl(const swr_problem_t* p, int64_t t0, const void* x, const void* a, const void* b,
              const void* c, void* y, float* state, bool exact, void* stream) {
    Resolved r;
    int rc = resolve(p, &r);
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    if (t0 < 0) return SWR_ERR_SHAPE;
    const int64_t seqs = p->B * p->H;
    if (seqs == 0 || p->T == 0) return SWR_OK;   // no token: the state is unchanged
    if (!x || !a || !b || !c || !y || !state) return SWR_ERR_NULL;
    const int64_t vb = step_vbytes(p, r);
    for (const void* q : {x, b, c, (const void*)y})
        if (!aligned(q, vb)) return SWR_ERR_ALIGN;
    if (!aligned(a, r.pc ? vb : r.es) || !aligned(state, 16)) return SWR_ERR_ALIGN;
    if ((rc = check_step_strides(p, r, vb)) != SWR_OK) return rc;
    const int64_t sbytes = seqs * p->D * 4 * (exact ? 1 : 2);
    const Span ins[4] = {span(x, r.xspan), span(b, r.xspan), span(c, r.xspan), span(a, r.aspan * r.es)};
    const Span sy = span(y, r.xspan), ss = span(state, sbytes);
    for (const Span& s : ins)
        if (overlap(sy, s) || overlap(ss, s)) return SWR_ERR_ALIAS;
    if (overlap(sy, ss)) return SWR_ERR_ALIAS;

    swr::StepParams q{};
    q.x = x; q.a = a; q.b = b; q.c = c; q.y = y; q.state = state;
    q.B = p->B; q.K = p->T; q.H = p->H;
    q.sx_b = p->sx_b; q.sx_t = p->sx_t; q.sx_h = p->sx_h;
    q.sa_b = p->sa_b; q.sa_t = p->sa_t; q.sa_h = p->sa_h;
    q.t0 = t0;
    q.block = (int32_t)p->block;
    q.residual = (p->flags & SWR_FLAG_RESIDUAL) ? 1 : 0;
    q.sig_a = (p->flags & SWR_FLAG_SIGMOID_DECAY) ? 1 : 0;
    q.sig_b = (p->flags & SWR_FLAG_SIGMOID_PREGATE) ? 1 : 0;
    return swr::launch_step(q, p->dtype, (int)p->D, exact, r.pc, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

}  // namespace

extern "C" {

int swr_step(const swr_problem_t* problem, int64_t t0, const void* x, const void* a, const void* b,
             const void* c, void* y, float* state, void* stream) {
    return step_impl(problem, t0, x, a, b, c, y, state, false, stream);
}

int swr_exact_step(const swr_problem_t* problem, const void* x, const void* a, const void* b,
                   const void* c, void* y, float* state, void* stream) {
    return step_impl(problem, 0, x, a, b, c, y, state, true, stream);
}

int swr_decode_state(const swr_problem_t* p, const void* a, const float* carriers, float* state,
                     void* stream) {
    Resolved r;
    const int rc = resolve(p, &r);
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    const int64_t seqs = p->B * p->H;
    if (seqs == 0) return SWR_OK;
    if (!state || (p->T > 0 && (!a || !carriers))) return SWR_ERR_NULL;
    const int64_t vb = step_vbytes(p, r);
    if (!aligned(state, 16) || (carriers && !aligned(carriers, 16))) return SWR_ERR_ALIGN;
    if (p->T > 0) {
        if (!aligned(a, r.pc ? vb : r.es)) return SWR_ERR_ALIGN;
        if (r.pc && check_step_strides(p, r, vb) != SWR_OK) return SWR_ERR_ALIGN;
    }
    const Span ss = span(state, seqs * 2 * p->D * 4);
    if (overlap(ss, span(a, r.aspan * r.es)) || overlap(ss, span(carriers, r.carriers * 4)))
        return SWR_ERR_ALIAS;

    swr::StateParams q{};
    q.a = a; q.carriers = carriers; q.state = state;
    q.B = p->B; q.T = p->T; q.H = p->H;
    q.sa_b = r.pc ? p->sx_b : p->sa_b;
    q.sa_t = r.pc ? p->sx_t : p->sa_t;
    q.sa_h = r.pc ? p->sx_h : p->sa_h;
    q.nblocks = r.nblocks;
    q.lshift = p->block == 16 ? 4 : p->block == 32 ? 5 : p->block == 64 ? 6 : 7;
    q.sig_a = (p->flags & SWR_FLAG_SIGMOID_DECAY) ? 1 : 0;
    return swr::launch_state(q, p->dtype, (int)p->D, r.pc, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Uniform window
// ---------------------------------------------------------------------------

namespace {

// Launch plan of the uniform-window kernels: heads of more than 64 channels
// run as 64-channel virtual heads; a workgroup holds 8 waves, one per
// sub-block of a block, times 128 / block virtual heads.
struct UniPlan {
    Resolved r;         // shape, stride and size validation shared with the jagged window
    int hshift, dk, cpl;
    int64_t hv, vbytes, run_len, nruns, nwork;
};

int uni_resolve(const swr_problem_t* p, UniPlan* u, bool backward) {
    int rc = resolve(p, &u->r, false);
    if (rc != SWR_OK) return rc;
    if (!u->r.natural) return SWR_ERR_UNSUPPORTED;
    if (p->flags & SWR_FLAG_PER_CHANNEL_DECAY) return SWR_ERR_UNSUPPORTED;
    u->hshift = p->D > 64 ? 1 : 0;
    u->dk = (int)(p->D >> u->hshift);
    u->cpl = u->dk / 16;
    u->hv = p->H << u->hshift;
    u->vbytes = std::min<int64_t>(16, (int64_t)u->cpl * u->r.es);
    const int64_t hw = 128 / p->block;                   // virtual heads per workgroup
    const int64_t groups = p->B * ((u->hv + hw - 1) / hw);
    if (u->r.empty) {
        u->run_len = p->block;
        u->nruns = u->nwork = 0;
        return SWR_OK;
    }
    // The backward: one 8-wave workgroup per compute unit.  The forward: runs
    // between those of about 2048 and about 512 workgroups, as close to 2048
    // tokens as that allows (measured on MI355X against 512 workgroups:
    // B8 T16384 H16 d128 455 -> 438 us, B1 T131072 H32 d64 466 -> 449, B16
    // T8192 H32 d64 426 -> 423).
    if (p->run_len > 0)
        u->run_len = p->run_len;
    else if (backward)
        u->run_len = pick_run_len(p->T, groups, p->block, 256);
    else
        u->run_len = std::max(pick_run_len(p->T, groups, p->block, 2048),
                              std::min<int64_t>(2048, pick_run_len(p->T, groups, p->block, 512)));
    u->nruns = (p->T + u->run_len - 1) / u->run_len;
    if (u->nruns > kMaxWorkgroups / groups) return SWR_ERR_UNSUPPORTED;
    u->nwork = groups * u->nruns;
    return SWR_OK;
}

int uni_check_strides(const swr_problem_t* p, const UniPlan& u) {
    const Dim xd[3] = {{p->B, p->sx_b}, {p->T, p->sx_t}, {p->H, p->sx_h}};
    for (const Dim& d : xd)
        if (d.size > 1 && (d.stride * u.r.es) % u.vbytes != 0) return SWR_ERR_ALIGN;
    return SWR_OK;
}

swr::Params uni_params(const swr_problem_t* p, const UniPlan& u) {
    swr::Params k = make_params(p, u.r, false);
    k.Hv = u.hv;
    k.hshift = u.hshift;
    k.run_len = u.run_len;
    k.nruns = u.nruns;
    k.nwork = u.nwork;
    return k;
}

}  // namespace

extern "C" {

int swr_uniform_forward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                        const void* c, void* y, void* stream) {
    UniPlan u;
    int rc = uni_resolve(p, &u, false);
    if (rc != SWR_OK) return rc;
    if (u.r.empty) return SWR_OK;
    if (!x || !a || !b || !c || !y) return SWR_ERR_NULL;
    for (const void* q : {x, b, c, (const void*)y})
        if (!aligned(q, u.vbytes)) return SWR_ERR_ALIGN;
    if (!aligned(a, u.r.es)) return SWR_ERR_ALIGN;
    if ((rc = uni_check_strides(p, u)) != SWR_OK) return rc;
    const Span sy = span(y, u.r.xspan);
    for (const Span& s : {span(x, u.r.xspan), span(b, u.r.xspan), span(c, u.r.xspan), span(a, u.r.aspan * u.r.es)})
        if (overlap(sy, s)) return SWR_ERR_ALIAS;
    swr::Params k = uni_params(p, u);
    k.x = x; k.a = a; k.b = b; k.c = c; k.y = y;
    return swr::launch_uniform(k, p->dtype, u.cpl, false, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

int swr_uniform_backward(const swr_problem_t* p, const void* x, const void* a, const void* b,
                         const void* c, const void* dy, void* dx, float* da, void* db, void* dc,
                         void* stream) {
    UniPlan u;
    int rc = uni_resolve(p, &u, true);
    if (rc != SWR_OK) return rc;
    if (u.r.empty) return SWR_OK;
    if (!x || !a || !b || !c || !dy || !dx || !da || !db || !dc) return SWR_ERR_NULL;
    for (const void* q : {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc})
        if (!aligned(q, u.vbytes)) return SWR_ERR_ALIGN;
    if (!aligned(a, u.r.es) || !aligned(da, 4)) return SWR_ERR_ALIGN;
    if ((rc = uni_check_strides(p, u)) != SWR_OK) return rc;
    const Span outs[4] = {span(dx, u.r.xspan), span(db, u.r.xspan), span(dc, u.r.xspan),
                          span(da, u.r.aspan * 4)};
    const Span ins[5] = {span(x, u.r.xspan), span(b, u.r.xspan), span(c, u.r.xspan), span(dy, u.r.xspan),
                         span(a, u.r.aspan * u.r.es)};
    for (int i = 0; i < 4; ++i) {
        for (const Span& s : ins)
            if (overlap(outs[i], s)) return SWR_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], outs[j])) return SWR_ERR_ALIAS;
    }
    swr::Params k = uni_params(p, u);
    k.x = x; k.a = a; k.b = b; k.c = c; k.dy = dy;
    k.dx = dx; k.da = da; k.db = db; k.dc = dc;
    return swr::launch_uniform(k, p->dtype, u.cpl, true, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

int swr_uniform_launch_info(const swr_problem_t* problem, int64_t* fwd_run_len, int64_t* fwd_workgroups,
                            int64_t* bwd_run_len, int64_t* bwd_workgroups) {
    UniPlan f, b;
    int rc = uni_resolve(problem, &f, false);
    if (rc != SWR_OK) return rc;
    if ((rc = uni_resolve(problem, &b, true)) != SWR_OK) return rc;
    if (fwd_run_len) *fwd_run_len = f.run_len;
    if (fwd_workgroups) *fwd_workgroups = f.nwork;
    if (bwd_run_len) *bwd_run_len = b.run_len;
    if (bwd_workgroups) *bwd_workgroups = b.nwork;
    return SWR_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Gates shared by groups of heads
// ---------------------------------------------------------------------------

namespace {

// Validation common to both shared-gate calls: the problem as for the jagged
// window (no per-channel decay, no packing), then the group and the gate
// tensors' strides.  gspan receives the bytes spanned by one gate tensor.
int gates_resolve(const swr_problem_t* p, int64_t group, const int64_t* gst, Resolved* r, int64_t* gspan) {
    int rc = resolve(p, r, false);
    if (rc != SWR_OK) return rc;
    if (!r->natural) return SWR_ERR_UNSUPPORTED;
    if (p->flags & SWR_FLAG_PER_CHANNEL_DECAY) return SWR_ERR_UNSUPPORTED;
    if (group < 1 || (p->H > 0 && p->H % group != 0)) return SWR_ERR_SHAPE;
    *gspan = 0;
    if (r->empty) return SWR_OK;
    if (!gst) return SWR_ERR_NULL;
    Dim gd[4] = {{p->B, gst[0]}, {p->T, gst[1]}, {p->H / group, gst[2]}, {p->D, 1}};
    for (int i = 0; i < 3; ++i)
        if (gd[i].size > 1 && (gd[i].stride * r->es) % r->vbytes != 0) return SWR_ERR_ALIGN;
    const int64_t go = max_offset(gd, 4);
    if (go < 0 || !non_overlapping(gd, 4)) return SWR_ERR_SHAPE;   // (sorts gd)
    *gspan = (go + 1) * r->es;
    const int64_t lim = 0x7fffffffLL;   // 32-bit lane offsets over 16 rows
    if (gst[1] > (lim - p->D * r->es) / (16 * r->es)) return SWR_ERR_UNSUPPORTED;
    if (p->H * p->D > (lim - p->D * 4) / (16 * 4)) return SWR_ERR_UNSUPPORTED;
    return SWR_OK;
}

void set_gates(swr::Params* k, int64_t group, const int64_t* gst) {
    k->group = group;
    k->sg_b = gst[0]; k->sg_t = gst[1]; k->sg_h = gst[2];
}

}  // namespace

extern "C" {

int64_t swr_shared_gates_workspace_bytes(const swr_problem_t* p, int64_t group) {
    Resolved r;
    const int rc = resolve(p, &r, false);
    if (rc != SWR_OK) return rc;
    if (!r.natural) return SWR_ERR_UNSUPPORTED;
    if (group < 1 || (p->H > 0 && p->H % group != 0)) return SWR_ERR_SHAPE;
    // groups of up to grouped_max_heads() heads are summed inside the backward
    return group <= swr::grouped_max_heads() ? 0 : 2 * p->B * p->T * p->H * p->D * 4;
}

int swr_forward_shared_gates(const swr_problem_t* p, int64_t group, const int64_t* gate_strides,
                             const void* x, const void* a, const void* b, const void* c, void* y,
                             float* carriers, void* stream) {
    Resolved r;
    int64_t gspan;
    int rc = gates_resolve(p, group, gate_strides, &r, &gspan);
    if (rc != SWR_OK) return rc;
    if (r.empty) return SWR_OK;
    if (!x || !a || !b || !c || !y) return SWR_ERR_NULL;
    for (const void* q : {x, b, c, (const void*)y})
        if (!aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
    if (!aligned(a, r.es) || (carriers && !aligned(carriers, 16))) return SWR_ERR_ALIGN;
    if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    const Span ins[4] = {span(x, r.xspan), span(b, gspan), span(c, gspan), span(a, r.aspan * r.es)};
    const Span sy = span(y, r.xspan), sv = span(carriers, carriers ? r.carriers * 4 : 0);
    for (const Span& s : ins)
        if (overlap(sy, s) || overlap(sv, s)) return SWR_ERR_ALIAS;
    if (overlap(sy, sv)) return SWR_ERR_ALIAS;
    swr::Params k = make_params(p, r, false);
    set_gates(&k, group, gate_strides);
    k.x = x; k.a = a; k.b = b; k.c = c; k.y = y; k.carriers = carriers;
    return swr::launch(k, p->dtype, r.dk, r.fwd, false, false, 1, swr::kGrouped, stream) == hipSuccess
               ? SWR_OK : SWR_ERR_HIP;
}

int swr_backward_shared_gates(const swr_problem_t* p, int64_t group, const int64_t* gate_strides,
                              const void* x, const void* a, const void* b, const void* c, const void* dy,
                              const float* carriers, void* dx, float* da, void* db, void* dc,
                              void* workspace, void* stream) {
    Resolved r;
    int64_t gspan;
    int rc = gates_resolve(p, group, gate_strides, &r, &gspan);
    if (rc != SWR_OK) return rc;
    if (r.empty) return SWR_OK;
    const bool fused = group <= swr::grouped_max_heads();
    if (!x || !a || !b || !c || !dy || !carriers || !dx || !da || !db || !dc || (!fused && !workspace))
        return SWR_ERR_NULL;
    for (const void* q : {x, b, c, dy, (const void*)dx, (const void*)db, (const void*)dc})
        if (!aligned(q, r.vbytes)) return SWR_ERR_ALIGN;
    if (!aligned(a, r.es) || !aligned(da, 4) || !aligned(carriers, 16) || !aligned(workspace, 16))
        return SWR_ERR_ALIGN;
    if ((rc = check_strides_aligned(p, r)) != SWR_OK) return rc;
    const int64_t wbytes = fused || !workspace ? 0 : 2 * p->B * p->T * p->H * p->D * 4;
    const Span outs[5] = {span(dx, r.xspan), span(db, gspan), span(dc, gspan), span(da, r.aspan * 4),
                          span(workspace, wbytes)};
    const Span ins[6] = {span(x, r.xspan), span(b, gspan), span(c, gspan), span(dy, r.xspan),
                         span(a, r.aspan * r.es), span(carriers, r.carriers * 4)};
    for (int i = 0; i < 5; ++i) {
        for (const Span& s : ins)
            if (overlap(outs[i], s)) return SWR_ERR_ALIAS;
        for (int j = i + 1; j < 5; ++j)
            if (overlap(outs[i], outs[j])) return SWR_ERR_ALIAS;
    }
    swr::Params k = make_params(p, r, true);
    set_gates(&k, group, gate_strides);
    k.x = x; k.a = a; k.b = b; k.c = c; k.dy = dy;
    k.dx = dx; k.da = da; k.db = db; k.dc = dc;
    k.carriers = const_cast<float*>(carriers);
    if (fused) {
        // one workgroup per (batch, group, 64-channel half, run), whole blocks per step
        k.hshift = p->D > 64 ? 1 : 0;
        k.Hv = (p->H / group) << k.hshift;
        const int64_t units = p->B * k.Hv;
        const int tw = p->block >= 128 ? 8 : 4;
        k.run_len = p->run_len > 0 ? p->run_len : pick_run_len(p->T, units, 16 * tw, 256);
        k.nruns = (p->T + k.run_len - 1) / k.run_len;
        if (k.nruns > kMaxWorkgroups / units) return SWR_ERR_UNSUPPORTED;
        k.nwork = units * k.nruns;
        const int cpl = (int)(std::min<int64_t>(p->D, 64) / 16);
        return swr::launch_grouped_backward(k, p->dtype, cpl, tw, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
    }
    k.gws = (float*)workspace;
    if (swr::launch(k, p->dtype, r.dk, r.bwd, true, false, 1, swr::kGrouped, stream) != hipSuccess)
        return SWR_ERR_HIP;
    return swr::launch_gate_reduce(k, p->dtype, (int)p->D, stream) == hipSuccess ? SWR_OK : SWR_ERR_HIP;
}

}  // extern "C"
