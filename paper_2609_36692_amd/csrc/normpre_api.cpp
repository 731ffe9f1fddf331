// Host side of the NormPre C ABI (include/normpre.h): argument validation,
// grouping of equal shapes into batched launches, the device workspace, and
// the launch sequence of one optimizer step (Alg. 1 of the paper, with
// Newton-Schulz for NormPre-G and Alg. 2, the randomized interaction sketch,
// for NormPre-L).  Every numerical step runs in the gfx950 kernels of this
// library; nothing here computes on the host.
#include "../../include/normpre.h"
#include "np_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

using namespace np;

namespace {

thread_local std::string g_noctx_error;

constexpr int64_t kMaxDim = int64_t(1) << 20;
constexpr int64_t kMaxElems = int64_t(1) << 31;
constexpr int kMaxRowLen = 32768;   // row-active register kernel limit
constexpr int kMaxEll = 384;
// Widths of Gamma_Q above this go to the dense eigensolver (tridiagonal
// reduction, bisection, inverse iteration) instead of the Jacobi kernels.
constexpr int kEigJacobiMax = 104;
// Exact NormPre-L above kMaxEll active rows: dense fp64 eigensolver on the
// a x a interaction matrix (tridiagonal reduction, bisection, inverse
// iteration), up to this many active rows.
constexpr int64_t kMaxExactRows = 8192;
constexpr int kColRowChunk = 128;   // rows per block in the column-active pass
constexpr int kMaxSplits = 16;
constexpr int kEigSweeps = 30;
// NormPre-L: largest share of ||Psi||_F^2 in the selected modes for which
// ||T||_F^2 is taken in closed form (see sketch_back).
constexpr float kClosedNormFrac = 0.25f;
constexpr size_t kGroupBudget = size_t(24) << 30;  // workspace bytes per item
constexpr size_t kRoundBudget = size_t(48) << 30;  // workspace bytes per round
// Static scratch of normpre_step_noalloc(): the whole workspace of that entry
// point (items and rounds are cut to fit it).  Every device that loads the
// library holds one copy for the life of the process.
constexpr size_t kScratchBytes = size_t(256) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];
static_assert(kScratchBytes == (size_t)NORMPRE_NOALLOC_SCRATCH_BYTES, "scratch size differs from the header");

struct Fail {
    int code;
    std::string msg;
};

std::string fmt(const char* f, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, f);
    vsnprintf(buf, sizeof buf, f, ap);
    va_end(ap);
    return buf;
}

int orientation_of(const normpre_hparams& hp) {
    if (hp.orientation == NORMPRE_ORIENT_ROW) return 0;
    if (hp.orientation == NORMPRE_ORIENT_COL) return 1;
    return (int)(((hp.step % 2) + 2) % 2);
}

// Exact NormPre-L through the dense eigensolver (more than kMaxEll active rows).
bool exact_large(const normpre_hparams& hp, int64_t active_rows) {
    return (hp.flags & NORMPRE_FLAG_L_EXACT) && active_rows > kMaxEll;
}

// l of Alg. 2.  The exact variant spans all active rows, or, above kMaxEll
// of them, the leading min(r, a) eigenvectors of Gamma (all the selected
// modes can come from).
int sketch_width(const normpre_hparams& hp, int64_t active_rows) {
    if (exact_large(hp, active_rows)) return (int)std::min<int64_t>(active_rows, hp.rank);
    if (hp.flags & NORMPRE_FLAG_L_EXACT) return (int)std::min<int64_t>(active_rows, INT32_MAX);
    return (int)std::min<int64_t>(active_rows, (int64_t)hp.rank + hp.oversample);
}

int power_iterations(const normpre_hparams& hp) {
    return (hp.flags & NORMPRE_FLAG_L_EXACT) ? 0 : hp.power_iters;
}

// Active orientation of the step; the Muon reference step has none (it
// works on the whole matrix in the W layout).
int step_orientation(int variant, const normpre_hparams& hp) {
    return variant == NORMPRE_VARIANT_MUON ? 0 : orientation_of(hp);
}

int tangent_mode(const normpre_hparams& hp) {
    if (hp.flags & NORMPRE_FLAG_TANGENT_NONE) return np::kTangentNone;
    if (hp.flags & NORMPRE_FLAG_TANGENT_STRICT) return np::kTangentStrict;
    return np::kTangentRelaxed;
}

// Shared by normpre_validate() and normpre_step().
Fail validate(int variant, int num_mats, const int64_t* shapes, const normpre_hparams* hp) {
    if (variant < NORMPRE_VARIANT_G || variant > NORMPRE_VARIANT_NORMALIZE_ONLY)
        return {NORMPRE_ERR_INVALID_ARG, fmt("unknown variant %d", variant)};
    if (num_mats < 0) return {NORMPRE_ERR_INVALID_ARG, "num_mats < 0"};
    if (!hp) return {NORMPRE_ERR_INVALID_ARG, "hparams is null"};
    if (num_mats > 0 && !shapes) return {NORMPRE_ERR_INVALID_ARG, "shapes is null"};
    if (!std::isfinite(hp->lr) || hp->lr < 0.f) return {NORMPRE_ERR_INVALID_ARG, "lr must be finite and >= 0"};
    if (!std::isfinite(hp->momentum)) return {NORMPRE_ERR_INVALID_ARG, "momentum must be finite"};
    if (!std::isfinite(hp->weight_decay) || hp->weight_decay < 0.f)
        return {NORMPRE_ERR_INVALID_ARG, "weight_decay must be finite and >= 0"};
    if (!std::isfinite(hp->target_rms)) return {NORMPRE_ERR_INVALID_ARG, "target_rms must be finite"};
    if (!(hp->norm_eps > 0.f) || !std::isfinite(hp->norm_eps))
        return {NORMPRE_ERR_INVALID_ARG, "norm_eps must be finite and > 0"};
    if (hp->orientation < NORMPRE_ORIENT_ALTERNATING || hp->orientation > NORMPRE_ORIENT_BOTH)
        return {NORMPRE_ERR_INVALID_ARG, fmt("unknown orientation mode %d", hp->orientation)};
    if (hp->flags & ~(NORMPRE_FLAG_DEBUG | NORMPRE_FLAG_TIME_KERNELS | NORMPRE_FLAG_TANGENT_NONE |
                      NORMPRE_FLAG_TANGENT_STRICT | NORMPRE_FLAG_L_EXACT | NORMPRE_FLAG_SOURCE_X |
                      NORMPRE_FLAG_CHECK_FINITE))
        return {NORMPRE_ERR_INVALID_ARG, fmt("unknown flags 0x%x", hp->flags)};
    if ((hp->flags & NORMPRE_FLAG_CHECK_FINITE) && variant == NORMPRE_VARIANT_MUON)
        return {NORMPRE_ERR_INVALID_ARG, "NORMPRE_FLAG_CHECK_FINITE applies to the normalized variants"};
    if ((hp->flags & NORMPRE_FLAG_TANGENT_NONE) && (hp->flags & NORMPRE_FLAG_TANGENT_STRICT))
        return {NORMPRE_ERR_INVALID_ARG, "at most one tangent mode flag"};
    if ((hp->flags & NORMPRE_FLAG_L_EXACT) && variant != NORMPRE_VARIANT_L)
        return {NORMPRE_ERR_INVALID_ARG, "NORMPRE_FLAG_L_EXACT applies to NormPre-L only"};
    if ((hp->flags & NORMPRE_FLAG_SOURCE_X) && variant != NORMPRE_VARIANT_L)
        return {NORMPRE_ERR_INVALID_ARG, "NORMPRE_FLAG_SOURCE_X applies to NormPre-L only"};
    if ((hp->flags & NORMPRE_FLAG_SOURCE_X) && hp->orientation == NORMPRE_ORIENT_BOTH)
        return {NORMPRE_ERR_INVALID_ARG, "NORMPRE_FLAG_SOURCE_X needs a single active side"};
    if (variant == NORMPRE_VARIANT_G || variant == NORMPRE_VARIANT_MUON) {
        if (hp->ns_iters < 1 || hp->ns_iters > 64)
            return {NORMPRE_ERR_INVALID_ARG, fmt("ns_iters %d outside 1..64", hp->ns_iters)};
        for (int i = 0; i < 3; ++i)
            if (!std::isfinite(hp->ns_coeffs[i])) return {NORMPRE_ERR_INVALID_ARG, "ns_coeffs must be finite"};
        if (!std::isfinite(hp->ns_eps) || hp->ns_eps < 0.f)
            return {NORMPRE_ERR_INVALID_ARG, "ns_eps must be finite and >= 0"};
    } else if (variant == NORMPRE_VARIANT_L) {
        if (hp->rank < 1) return {NORMPRE_ERR_INVALID_ARG, fmt("rank %d < 1", hp->rank)};
        if (hp->oversample < 0) return {NORMPRE_ERR_INVALID_ARG, fmt("oversample %d < 0", hp->oversample)};
        if (hp->power_iters < 0 || hp->power_iters > 8)
            return {NORMPRE_ERR_INVALID_ARG, fmt("power_iters %d outside 0..8", hp->power_iters)};
    }
    const int k = step_orientation(variant, *hp);
    for (int i = 0; i < num_mats; ++i) {
        const int64_t m = shapes[2 * i], n = shapes[2 * i + 1];
        if (m < 1 || n < 1)
            return {NORMPRE_ERR_INVALID_ARG, fmt("matrix %d has shape %lld x %lld", i, (long long)m, (long long)n)};
        if (m > kMaxDim || n > kMaxDim || m * n > kMaxElems)
            return {NORMPRE_ERR_UNSUPPORTED, fmt("matrix %d (%lld x %lld) is too large", i, (long long)m, (long long)n)};
        const bool rows_pass = k == 0 || hp->orientation == NORMPRE_ORIENT_BOTH;
        if (rows_pass && n > kMaxRowLen && variant != NORMPRE_VARIANT_MUON)
            return {NORMPRE_ERR_UNSUPPORTED,
                    fmt("matrix %d: row-active rows of %lld elements exceed %d", i, (long long)n, kMaxRowLen)};
        if (variant == NORMPRE_VARIANT_L) {
            const int64_t a = k == 0 ? m : n;
            if (exact_large(*hp, a) && a > kMaxExactRows)
                return {NORMPRE_ERR_UNSUPPORTED,
                        fmt("matrix %d: exact NormPre-L on %lld active rows exceeds %lld", i, (long long)a,
                            (long long)kMaxExactRows)};
            const int64_t ell = sketch_width(*hp, a);
            if (ell > kMaxEll)
                return {NORMPRE_ERR_UNSUPPORTED,
                        fmt("matrix %d: %s %lld exceeds %d", i,
                            (hp->flags & NORMPRE_FLAG_L_EXACT) ? "exact NormPre-L with rank" : "sketch width",
                            (long long)ell, kMaxEll)};
        }
    }
    return {NORMPRE_OK, ""};
}

// -------------------------------------------------------------- timing ---
struct KStat {
    int64_t launches = 0;
    double ms = 0, flops = 0, bytes = 0, exec_flops = 0;
};
struct PendingEvent {
    int kclass;
    hipEvent_t start, stop;
    double flops, bytes, exec_flops;
};

struct DebugMat {
    int64_t rows = 0, cols = 0;
    int variant = 0, k = 0, ell = 0, top = 0;
    float* psi32 = nullptr;    // rows*cols
    float* t32 = nullptr;      // rows*cols (G)
    float* scalars = nullptr;  // [0] = ||T||^2, [1] = nsel (as int bits), ritz from [2]
};

}  // namespace

struct normpre_ctx {
    int device = 0;
    std::string err;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    hipStream_t last_stream = nullptr;
    bool have_stream = false;
    // debug state of the last step made with NORMPRE_FLAG_DEBUG
    std::vector<DebugMat> dbg;
    void* dbg_mem = nullptr;
    size_t dbg_bytes = 0;
    bool dbg_valid = false;
    hipStream_t dbg_stream = nullptr;
    // per-kernel timing
    KStat stats[NORMPRE_KCLASS_COUNT];
    std::vector<PendingEvent> pending;
    std::vector<hipEvent_t> event_pool;
    bool timing = false;
    hipStream_t stream = nullptr;
    // Orders a step after the previous step's work when the caller switches
    // streams (created by normpre_init, so no step allocates it).
    hipEvent_t order_ev = nullptr;
    // Workspace reserved by normpre_reserve(): steps then never grow it.
    bool reserved = false;
    // Non-finite counts of the last step made with NORMPRE_FLAG_CHECK_FINITE
    // (device, in that step's workspace; null after any other step).
    long long* status = nullptr;
    int status_count = 0;
    hipStream_t status_stream = nullptr;
    // Device address of the static scratch array of normpre_step_noalloc()
    // on this context's device (from hipGetSymbolAddress at init).
    void* scratch = nullptr;
};

namespace {

int set_err(normpre_ctx* ctx, int code, const std::string& msg) {
    if (ctx) ctx->err = msg;
    else g_noctx_error = msg;
    return code;
}

int hip_fail(normpre_ctx* ctx, hipError_t e, const char* what) {
    return set_err(ctx, NORMPRE_ERR_HIP, fmt("%s: %s", what, hipGetErrorString(e)));
}

hipEvent_t get_event(normpre_ctx* ctx) {
    if (!ctx->event_pool.empty()) {
        hipEvent_t e = ctx->event_pool.back();
        ctx->event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Runs one launch; with kernel timing on, times it with an event pair.  A
// GEMM launch takes the pair itself (recorded at the kernel's own start and
// end); any other launch is bracketed by stream-ordered records.
// `exec_flops`: MFMA work the launch issues (tiles x tile FLOPs, zero padding
// included); negative for launches that are not matrix products.
template <class F>
hipError_t timed(normpre_ctx* ctx, int kclass, double flops, double bytes, F&& launch, double exec_flops = -1.0) {
    if (!ctx->timing) return launch();
    hipEvent_t a = get_event(ctx), b = get_event(ctx);
    if (!a || !b) return hipErrorOutOfMemory;
    hipError_t e = hipEventRecord(a, ctx->stream);
    if (e != hipSuccess) return e;
    np::arm_launch_events(a, b);
    e = launch();
    const bool unused = np::disarm_launch_events();
    if (e != hipSuccess) return e;
    if (unused) {
        e = hipEventRecord(b, ctx->stream);
        if (e != hipSuccess) return e;
    }
    ctx->pending.push_back({kclass, a, b, flops, bytes, exec_flops < 0.0 ? 0.0 : exec_flops});
    return hipSuccess;
}

int collect_events(normpre_ctx* ctx) {
    for (auto& p : ctx->pending) {
        hipError_t e = hipEventSynchronize(p.stop);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, p.start, p.stop);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventElapsedTime");
        KStat& s = ctx->stats[p.kclass];
        s.launches += 1;
        s.ms += ms;
        s.flops += p.flops;
        s.bytes += p.bytes;
        s.exec_flops += p.exec_flops;
        ctx->event_pool.push_back(p.start);
        ctx->event_pool.push_back(p.stop);
    }
    ctx->pending.clear();
    return NORMPRE_OK;
}

// Bump allocator over the workspace (256-byte aligned slices).
struct Arena {
    char* base;
    size_t off = 0;
    size_t cap;
    template <class T>
    T* take(int64_t count) {
        off = (off + 255) & ~size_t(255);
        T* p = reinterpret_cast<T*>(base ? base + off : nullptr);
        off += (size_t)count * sizeof(T);
        return p;
    }
};

struct Group {
    int64_t m, n;
    std::vector<int> idx;   // positions in the caller's list
};

// Workspace layout of one group; with base == nullptr it only measures.
struct GWork {
    // shared
    half_t* psi;
    // L with the interaction source X: trace-matched X (fp16, W layout),
    // the active rows' ||x_i||^2 and the per-matrix sum (2 floats).
    half_t* xs;
    float* xsq;
    float* xtot;
    float* psisq;
    float* scale;
    double* colpart;
    // G
    half_t* xb;
    half_t* amat;
    half_t* bmat;
    float* sumsq;           // per-tile partial sums of T^2 (both variants)
    int* nfin;              // finite check: non-finite count slots
    float* tn2;             // per-matrix ||T||_F^2
    // L
    half_t* omega;
    half_t* v16[2];
    float* v32[2];
    float* part;
    double* gpart;
    double* chol;
    float* rinv;
    float* kmat;
    half_t* qlen;
    half_t* flen;
    float* eigs;
    float* ritz;
    int* nsel;
    int* lneed;             // NormPre-L: 1 where ||T||_F needs the norm pass
    // exact NormPre-L above kMaxEll active rows
    float* gam32;           // Gamma, fp32 a_pad x a_pad
    TriWork tw;             // eigensolver workspace (order a)
    double* lam;            // leading ell eigenvalues
};

struct Dims {
    int64_t m, n, mp, np_, sp, lp_;
    int k;
    bool tall;
    // L
    int64_t a, b, a_pad, b_pad;
    int ell, ellp, top;
    bool xl;                // exact NormPre-L through the dense eigensolver
};

Dims dims_of(int64_t m, int64_t n, int k, const normpre_hparams& hp) {
    Dims d;
    d.m = m;
    d.n = n;
    d.mp = round_up(m, kPad);
    d.np_ = round_up(n, kPad);
    d.sp = std::min(d.mp, d.np_);
    d.lp_ = std::max(d.mp, d.np_);
    d.k = k;
    d.tall = m > n;
    d.a = k == 0 ? m : n;
    d.b = k == 0 ? n : m;
    d.a_pad = k == 0 ? d.mp : d.np_;
    d.b_pad = k == 0 ? d.np_ : d.mp;
    d.ell = sketch_width(hp, d.a);
    d.ellp = (int)round_up(d.ell, kEllPad);
    d.top = std::min(hp.rank, d.ell);
    d.xl = exact_large(hp, d.a);
    return d;
}

// Newton-Schulz in Gram space (NormPre-G and the Muon reference step).  Every
// iterate is X_k = Q_k X_0 with Q_k a polynomial in A_0 = X_0 X_0^T, and with
// P_k = a I + b A_k + c A_k^2 the recurrences Q_{k+1} = P_k Q_k and
// A_{k+1} = X_{k+1} X_{k+1}^T = P_k A_k P_k hold exactly (the P_k commute with
// A_k).  The iterations then run on s x s matrices and X is formed only at
// segment ends: X_3 = Q_3 X_0 (with a fresh Gram A_3, which bounds the fp16
// error growth of the s x s recurrences) and T = X_5 = Q_5 X_3.  Nominal
// FLOPs per matrix 8 s^2 L + 28 s^3 against 20 s^2 L + 10 s^3 for the plain
// iteration; used for the quintic's five iterations when L >= 2 s.
constexpr int kGnsIters = 5;
constexpr int kGnsRestart = 3;

bool gram_space_ns(int variant, const Dims& d, const normpre_hparams& hp) {
    if (variant != NORMPRE_VARIANT_G && variant != NORMPRE_VARIANT_MUON) return false;
    if (hp.ns_iters != kGnsIters) return false;
    return std::max(d.m, d.n) >= 2 * std::min(d.m, d.n);
}

// Length chunk of the fp64 Gram: >= 256 for parallel blocks and at most
// kGramChunks chunks (the consumers always sum kGramChunks slots).
int gram_chunk_len(int64_t len) {
    return (int)std::max<int64_t>(256, round_up((len + kGramChunks - 1) / kGramChunks, 64));
}

int ns_tiles(const Dims& d) { return (int)((d.mp / 128) * (d.np_ / 128)); }
// Tiles of the NormPre-L apply passes (64 x 128).
int apply_tiles(const Dims& d) { return (int)((d.mp / 64) * (d.np_ / 128)); }
int combine_tiles(const Dims& d, TileCfg cfg) {
    const int64_t t = cfg == TileCfg::Big256 ? 256 : 128;
    return (int)((d.mp / t) * (d.np_ / t));
}

// Split count for a skinny product with output length n_out and reduction
// length k_len: doubled until the launch has one block per CU (256) or the
// chunks get short.  More splits stream Psi with more blocks but cost a
// reduction launch; one split writes the result directly (on GPT-2 Small's
// NormPre-L step a 1024-block target measured 2.7% slower).
int pick_splits(int64_t tiles_per_mat, int count, int64_t k_len) {
    int splits = 1;
    while (splits < kMaxSplits && tiles_per_mat * count * splits < 256 && k_len / (64 * splits * 2) >= 4)
        splits *= 2;
    return splits;
}

// One batch of equal-shape matrices (a sub-range of a shape group).
struct Item {
    int g = 0;            // shape group
    int first = 0;        // first position in the group's list
    int count = 0;
    Dims d{};
    GWork w{};
    int pool = -1;        // pool of its small matrices
    int pool_off = 0;     // its first matrix inside the pool
    TileCfg ccfg = TileCfg::Big;   // tile of its Newton-Schulz combines
    bool gns = false;     // Newton-Schulz iterations carried in Gram space
};

// Small matrices shared by the items of a round that have the same width:
// the s x s Newton-Schulz matrices (NormPre-G, keyed by s) or the l x l
// sketch matrices (NormPre-L, keyed by l), so one launch covers all of them.
struct Pool {
    int64_t key = 0;
    int count = 0;
    int64_t sp = 0;
    int ell = 0, ellp = 0, top = 0;
    half_t* amat = nullptr;
    half_t* bmat = nullptr;
    // Gram-space Newton-Schulz: its items hold pool slots [0, gns_count);
    // Q (double buffered, qcur the current one) and the product R.
    int gns_count = 0;
    half_t* qmat[2] = {nullptr, nullptr};
    half_t* rmat = nullptr;
    int qcur = 0;
    double* gpart = nullptr;
    double* chol = nullptr;
    float* rinv = nullptr;
    float* kmat = nullptr;
    float* eigs = nullptr;
    float* ritz = nullptr;
    int* nsel = nullptr;
    // Ritz pairs through the dense eigensolver (l > kEigJacobiMax)
    TriWork tw{};
    double* lam = nullptr;
    float* zbuf = nullptr;
};

// Workspace options of a step: the interaction-source-X buffers and the
// non-finite count slots of the finite check.
constexpr int kOptSourceX = 1, kOptCheck = 2;
int step_opts(int variant, const normpre_hparams& hp) {
    int o = 0;
    if (variant == NORMPRE_VARIANT_L && (hp.flags & NORMPRE_FLAG_SOURCE_X)) o |= kOptSourceX;
    if (hp.flags & NORMPRE_FLAG_CHECK_FINITE) o |= kOptCheck;
    return o;
}

// Count slots per matrix of the finite check (an upper bound for both
// orientations: one per row, or one per 128-row chunk and 64-column block).
int64_t nfin_stride(const Dims& d) {
    return std::max<int64_t>(d.m, ((d.m + kColRowChunk - 1) / kColRowChunk) * ((d.n + 63) / 64));
}

void carve_item(Arena& ar, Item& it, int variant, int opts) {
    const bool source_x = (opts & kOptSourceX) != 0;
    const Dims& d = it.d;
    const int count = it.count;
    GWork& w = it.w;
    const int64_t mn = d.mp * d.np_;
    w.psi = ar.take<half_t>(count * mn);
    w.psisq = ar.take<float>(count * d.lp_);
    w.scale = ar.take<float>(count * 2);
    w.colpart = ar.take<double>(count * normalize_cols_partials((int)d.m, (int)d.np_, kColRowChunk));
    w.sumsq = ar.take<float>(count * std::max(ns_tiles(d), apply_tiles(d)));
    w.tn2 = ar.take<float>(count);
    if (opts & kOptCheck) w.nfin = ar.take<int>(count * nfin_stride(d));
    if (variant == NORMPRE_VARIANT_G || variant == NORMPRE_VARIANT_MUON) {
        w.xb = ar.take<half_t>(count * mn);
    } else if (variant == NORMPRE_VARIANT_L) {
        const int64_t lp = d.ellp, maxpad = d.lp_;
        // Every l-major skinny buffer (Omega^T included) has the per-matrix
        // stride lp * maxpad that the sketch products assume.
        w.omega = ar.take<half_t>(count * lp * maxpad);
        for (int i = 0; i < 2; ++i) {
            w.v16[i] = ar.take<half_t>(count * lp * maxpad);
            w.v32[i] = ar.take<float>(count * lp * maxpad);
        }
        w.part = ar.take<float>(count * (int64_t)kMaxSplits * lp * maxpad);
        w.qlen = ar.take<half_t>(count * d.a_pad * lp);
        w.flen = ar.take<half_t>(count * d.b_pad * lp);
        w.lneed = ar.take<int>(count);
        if (d.xl) {
            const int64_t a = d.a;
            w.gam32 = ar.take<float>(count * d.a_pad * d.a_pad);
            w.tw.A = ar.take<float>(count * a * a);
            w.tw.vec = ar.take<double>(count * 4 * a);
            w.tw.d = ar.take<double>(count * a);
            w.tw.e = ar.take<double>(count * a);
            w.tw.tau = ar.take<double>(count * a);
            w.tw.lu = ar.take<double>(count * d.ell * 6 * a);
            w.tw.y = ar.take<double>(count * d.ell * a);
            w.lam = ar.take<double>(count * d.ell);
        }
        if (source_x) {
            w.xs = ar.take<half_t>(count * mn);
            w.xsq = ar.take<float>(count * d.lp_);
            w.xtot = ar.take<float>(count * 2);
        }
    }
}

void carve_pool(Arena& ar, Pool& p, int variant) {
    const int64_t c = p.count;
    if (variant == NORMPRE_VARIANT_G || variant == NORMPRE_VARIANT_MUON) {
        p.amat = ar.take<half_t>(c * p.sp * p.sp);
        p.bmat = ar.take<half_t>(c * p.sp * p.sp);
        if (p.gns_count > 0) {
            const int64_t gc = p.gns_count;
            p.qmat[0] = ar.take<half_t>(gc * p.sp * p.sp);
            p.qmat[1] = ar.take<half_t>(gc * p.sp * p.sp);
            p.rmat = ar.take<half_t>(gc * p.sp * p.sp);
        }
    } else if (variant == NORMPRE_VARIANT_L) {
        const int64_t lp = p.ellp;
        p.gpart = ar.take<double>(c * kGramChunks * lp * lp);
        p.chol = ar.take<double>(c * 2 * lp * lp);
        p.rinv = ar.take<float>(c * lp * lp);
        p.kmat = ar.take<float>(c * lp * lp);
        p.eigs = ar.take<float>(c * 2 * lp * lp);
        p.ritz = ar.take<float>(c * (int64_t)p.top);
        p.nsel = ar.take<int>(c);
        if (p.ell > kEigJacobiMax) {
            const int64_t n = p.ell, top = p.top;
            p.tw.A = ar.take<float>(c * n * n);
            p.tw.vec = ar.take<double>(c * 4 * n);
            p.tw.d = ar.take<double>(c * n);
            p.tw.e = ar.take<double>(c * n);
            p.tw.tau = ar.take<double>(c * n);
            p.tw.lu = ar.take<double>(c * top * 6 * n);
            p.tw.y = ar.take<double>(c * top * n);
            p.lam = ar.take<double>(c * top);
            p.zbuf = ar.take<float>(c * top * n);
        }
    }
}

// Assigns every item to the pool of its width; returns the pools.
std::vector<Pool> make_pools(std::vector<Item>& items, int variant) {
    std::vector<Pool> pools;
    for (Item& it : items) {
        const int64_t key = variant == NORMPRE_VARIANT_L ? it.d.ell : it.d.sp;
        int pi = -1;
        for (size_t q = 0; q < pools.size(); ++q)
            if (pools[q].key == key) pi = (int)q;
        if (pi < 0) {
            Pool p;
            p.key = key;
            p.sp = it.d.sp;
            p.ell = it.d.ell;
            p.ellp = it.d.ellp;
            p.top = it.d.top;
            pools.push_back(p);
            pi = (int)pools.size() - 1;
        }
        it.pool = pi;
    }
    // Gram-space items take the first slots of their pool, so their s x s
    // matrices form one contiguous range (one launch per Gram-space product).
    for (int pass = 0; pass < 2; ++pass)
        for (Item& it : items) {
            if (it.gns != (pass == 0)) continue;
            Pool& p = pools[it.pool];
            it.pool_off = p.count;
            p.count += it.count;
            if (it.gns) p.gns_count += it.count;
        }
    return pools;
}

// Carves a round's items and pools; with a null arena base it only measures.
size_t carve_round(Arena& ar, std::vector<Item>& items, std::vector<Pool>& pools, int variant, int opts) {
    for (Item& it : items) carve_item(ar, it, variant, opts);
    for (Pool& p : pools) carve_pool(ar, p, variant);
    return ar.off + 256;
}

size_t round_bytes(std::vector<Item> items, int variant, int opts) {
    std::vector<Pool> pools = make_pools(items, variant);
    Arena ar{nullptr, 0, 0};
    return carve_round(ar, items, pools, variant, opts);
}

struct StepCtx {
    normpre_ctx* ctx;
    hipStream_t s;
    const normpre_hparams* hp;
    float* const* W;
    const float* const* G;
    float* const* M;
    int variant;
    bool debug;
    const std::vector<Group>* groups;
    long long* status = nullptr;    // finite check: per-matrix counts, caller order
};


#define NP_TRY(expr, what)                                  \
    do {                                                    \
        hipError_t e__ = (expr);                            \
        if (e__ != hipSuccess) return hip_fail(sc.ctx, e__, what); \
    } while (0)

PtrChunk make_chunk(const StepCtx& sc, const std::vector<int>& idx, int begin, int cnt) {
    PtrChunk p{};
    for (int i = 0; i < cnt; ++i) {
        const int g = idx[begin + i];
        p.w[i] = sc.W[g];
        p.m[i] = sc.M[g];
        p.g[i] = sc.G[g];
    }
    return p;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

bool chunk_vec_ok(const PtrChunk& p, int cnt) {
    for (int i = 0; i < cnt; ++i)
        if (!aligned16(p.w[i]) || !aligned16(p.m[i]) || !aligned16(p.g[i])) return false;
    return true;
}

// Momentum + tangent + normalization for `count` matrices starting at
// position `first` of the group list, writing the group workspace.
int run_normalize(const StepCtx& sc, const Dims& d, const GWork& w, const std::vector<int>& idx, int first,
                  int count, DebugMat* dbg) {
    const int64_t mn = d.mp * d.np_;
    // Both axes: rows first, then the columns of the result (psisq then
    // holds the squared column norms).
    const bool both = sc.hp->orientation == NORMPRE_ORIENT_BOTH;
    const double bytes = 18.0 * (double)d.m * (double)d.n;
    for (int c0 = 0; c0 < count; c0 += kChunk) {
        const int cnt = std::min(kChunk, count - c0);
        NormArgs a{};
        a.ptrs = make_chunk(sc, idx, first + c0, cnt);
        a.rows = (int)d.m;
        a.cols = (int)d.n;
        a.ld_psi = d.np_;
        a.rows_pad = d.mp;
        a.psi = w.psi + (int64_t)c0 * mn;
        a.stride_psi = mn;
        a.psisq = w.psisq + (int64_t)c0 * d.lp_;
        a.stride_psisq = d.lp_;
        a.mu = sc.hp->momentum;
        a.eps = sc.hp->norm_eps;
        a.vec_ok = chunk_vec_ok(a.ptrs, cnt);
        a.tangent = tangent_mode(*sc.hp);
        if (w.xsq) a.xsq = w.xsq + (int64_t)c0 * d.lp_;
        if (w.nfin) {
            a.stride_nfin = nfin_stride(d);
            a.nfin = w.nfin + (int64_t)c0 * a.stride_nfin;
        }
        if (dbg) {
            // Debug copies are written chunk by chunk into per-matrix buffers
            // that are contiguous in the order of the caller's list.
            a.psi32 = dbg[idx[first + c0]].psi32;
            a.stride_psi32 = d.m * d.n;
            for (int i = 1; i < cnt; ++i)
                if (dbg[idx[first + c0 + i]].psi32 != a.psi32 + i * d.m * d.n) a.psi32 = nullptr;
            if (!a.psi32) return set_err(sc.ctx, NORMPRE_ERR_HIP, "internal: debug buffers not contiguous");
        }
        if (d.k == 0 || both) {
            NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE, 0.0, bytes * cnt,
                         [&] { return launch_normalize_rows(a, cnt, sc.s); }),
                   "normalize rows");
            if (both)
                NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE, 0.0, 6.0 * (double)d.m * (double)d.n * cnt,
                             [&] {
                                 return launch_psi_col_normalize(
                                     a, cnt,
                                     reinterpret_cast<float*>(
                                         w.colpart +
                                         (int64_t)c0 * normalize_cols_partials((int)d.m, (int)d.np_, kColRowChunk)),
                                     2 * normalize_cols_partials((int)d.m, (int)d.np_, kColRowChunk), kColRowChunk,
                                     sc.s);
                             }),
                       "normalize both axes");
        } else {
            NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE_COL, 0.0, bytes * cnt,
                         [&] {
                             return launch_normalize_cols(
                                 a, cnt,
                                 w.colpart + (int64_t)c0 * normalize_cols_partials((int)d.m, (int)d.np_, kColRowChunk),
                                 kColRowChunk, sc.s);
                         }),
                   "normalize cols");
        }
        if (a.nfin && sc.status) {
            IdxChunk ic{};
            for (int i = 0; i < cnt; ++i) ic.idx[i] = idx[first + c0 + i];
            const int64_t slots = nonfinite_slots(a, d.k == 0 || both, kColRowChunk);
            NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                         [&] { return launch_count_reduce(a.nfin, slots, a.stride_nfin, ic, cnt, sc.status, sc.s); }),
                   "non-finite counts");
        }
    }
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                 [&] {
                     return launch_psi_scale(w.psisq, d.lp_, both ? (int)d.n : (int)d.a, sc.hp->ns_eps, w.scale,
                                             count, sc.s);
                 }),
           "psi scale");
    if (w.xs) {
        // Interaction source X: X_s = sqrt(a / ||X||_F^2) D Psi, so that
        // X_s X_s^T is the trace-matched Gram of the active rows.
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                     [&] { return launch_psi_scale(w.xsq, d.lp_, (int)d.a, 0.f, w.xtot, count, sc.s); }),
               "x norm");
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE, 0.0, 4.0 * (double)d.mp * (double)d.np_ * count,
                     [&] {
                         return launch_source_x(w.psi, d.np_, mn, (int)d.m, (int)d.n, (int)d.mp, d.k, (int)d.a,
                                                w.xsq, d.lp_, w.xtot, w.xs, count, sc.s);
                     }),
               "source x");
    }
    return NORMPRE_OK;
}

// 256 x 256 tiles (8 waves) when a launch has enough of them to fill the
// 256 CUs, else 128 x 128 tiles.
// Muon reference input (Sec. 2.1): M <- mu M + G, ||M||_F, X0 = M / (||M||_F +
// ns_eps) in fp16 (W layout, zero padded).  The per-block sums of M^2 reuse
// the row-statistics buffer.
int run_muon_input(const StepCtx& sc, const Dims& d, const GWork& w, const std::vector<int>& idx, int first,
                   int count, DebugMat* dbg) {
    const int64_t mn = d.mp * d.np_;
    const int nblk = momentum_sumsq_blocks(d.m * d.n);
    if (nblk > d.lp_) return set_err(sc.ctx, NORMPRE_ERR_HIP, "internal: muon partial buffer too small");
    std::vector<NormArgs> chunks;
    for (int c0 = 0; c0 < count; c0 += kChunk) {
        const int cnt = std::min(kChunk, count - c0);
        NormArgs a{};
        a.ptrs = make_chunk(sc, idx, first + c0, cnt);
        a.rows = (int)d.m;
        a.cols = (int)d.n;
        a.ld_psi = d.np_;
        a.rows_pad = d.mp;
        a.psi = w.psi + (int64_t)c0 * mn;
        a.stride_psi = mn;
        a.mu = sc.hp->momentum;
        a.vec_ok = chunk_vec_ok(a.ptrs, cnt);
        if (dbg) {
            a.psi32 = dbg[idx[first + c0]].psi32;
            a.stride_psi32 = d.m * d.n;
            for (int i = 1; i < cnt; ++i)
                if (dbg[idx[first + c0 + i]].psi32 != a.psi32 + i * d.m * d.n) a.psi32 = nullptr;
            if (!a.psi32) return set_err(sc.ctx, NORMPRE_ERR_HIP, "internal: debug buffers not contiguous");
        }
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE, 0.0, 12.0 * (double)d.m * (double)d.n * cnt,
                     [&] { return launch_momentum_sumsq(a, cnt, w.psisq + (int64_t)c0 * d.lp_, d.lp_, sc.s); }),
               "muon momentum");
        chunks.push_back(a);
    }
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                 [&] { return launch_psi_scale(w.psisq, d.lp_, nblk, sc.hp->ns_eps, w.scale, count, sc.s); }),
           "muon scale");
    for (size_t c = 0; c < chunks.size(); ++c) {
        const int c0 = (int)c * kChunk, cnt = std::min(kChunk, count - c0);
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NORMALIZE, 0.0, (4.0 * d.m * d.n + 2.0 * mn) * cnt,
                     [&] { return launch_scaled_cast(chunks[c], cnt, w.scale + 2 * c0, sc.s); }),
               "muon cast");
    }
    return NORMPRE_OK;
}

// 256 x 256 tiles (8 waves, 1 block per CU) once a launch has enough of them
// to fill the chip several times over (symmetric products count their
// upper-triangle tiles); below that the 128 x 128 tile (2 blocks per CU)
// keeps more CUs busy.  Measured on random data: symmetric 1024^3 products
// x56 (560 large tiles) ran 648 TFLOP/s on the small tile against 584 on the
// large one, 2048^3 x84 (3024 large tiles) 717 against 740; the combine
// switches earlier (12-matrix launches: 432 large tiles faster than the
// small ones, 324 slower).  A long reduction (K >= 4096) amortizes the
// large tile's multi-pass epilogue, and there 512 tiles suffice: a single
// symmetric 8192^3 product (528 large tiles) runs ~15% faster on the large
// tile than on the small one.  `K` is the shortest reduction of the launch.
TileCfg ns_cfg(int64_t M, int64_t N, int64_t K, bool sym, int count) {
    const int64_t tm = M / 256, tn = N / 256;
    const int64_t tiles = (sym ? tm * (tm + 1) / 2 : tm * tn) * count;
    const int64_t sym_min = K >= 4096 ? 512 : 1024;
    return tiles >= (sym ? sym_min : 384) ? TileCfg::Big256 : TileCfg::Big;
}

// MFMA FLOPs a product launch issues for `count` matrices of M x N x K with
// tile `cfg`: symmetric products compute the upper-triangular tiles only.
double issued_flops(TileCfg cfg, int64_t M, int64_t N, int64_t K, bool sym, int64_t count) {
    const int64_t bm = gemm_tile_m(cfg), bn = gemm_tile_n(cfg);
    const int64_t tm = M / bm, tn = N / bn;
    const int64_t tiles = sym ? tm * (tm + 1) / 2 : tm * tn;
    return 2.0 * (double)tiles * (double)(bm * bn) * (double)K * (double)count;
}

// The Grams of every item of one pool with the same operand layout, in one
// launch: small same-s batches (e.g. the three wide shapes of a transformer
// block) fill the chip together where each alone would not.
int gram_pool_launch(const StepCtx& sc, std::vector<const Item*> its, const Pool& pl, int iter, bool first_it) {
    const int64_t ss = pl.sp * pl.sp;
    // Longest K first: the costly matrices start in the first wave of blocks
    // and the cheap ones fill the tail.
    std::stable_sort(its.begin(), its.end(), [](const Item* a, const Item* b) { return a->d.lp_ > b->d.lp_; });
    const int layout = its[0]->d.tall ? 2 : 0;
    GramGroups gg{};
    double flops = 0.0, bytes = 0.0;
    int total = 0;
    for (const Item* it : its) {
        const Dims& d = it->d;
        const int g = gg.n++;
        gg.zbeg[g] = total;
        gg.x[g] = (iter & 1) ? it->w.xb : it->w.psi;
        gg.ld[g] = d.np_;
        gg.stride[g] = d.mp * d.np_;
        gg.K[g] = (int)d.lp_;
        gg.mul[g] = first_it ? it->w.scale : nullptr;
        gg.zout[g] = it->pool_off;
        total += it->count;
        const double s_ = (double)std::min(d.m, d.n), l_ = (double)std::max(d.m, d.n);
        flops += 2.0 * s_ * s_ * l_ * it->count;
        bytes += 2.0 * (s_ * l_ + s_ * s_) * it->count;
    }
    gg.zbeg[gg.n] = total;
    EpiAffine e{};
    e.out = pl.amat; e.ld_out = pl.sp; e.stride_out = ss;
    e.mul_pow = first_it ? 2 : 0;
    e.ca = 1.f; e.cs = 0.f;
    int64_t kmin = its[0]->d.lp_;
    for (const Item* it : its) kmin = std::min(kmin, it->d.lp_);
    const TileCfg cfg = ns_cfg(pl.sp, pl.sp, kmin, true, total);
    double issued = 0.0;
    for (const Item* it : its) issued += issued_flops(cfg, pl.sp, pl.sp, it->d.lp_, true, it->count);
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NS_GRAM, flops, bytes,
                 [&] { return launch_gemm_gram_grouped(cfg, layout, gg, (int)pl.sp, e, sc.s); }, issued),
           "ns gram");
    return NORMPRE_OK;
}

int gram_launches(const StepCtx& sc, const std::vector<Item>& items, const std::vector<Pool>& pools, int iter,
                  bool first_it) {
    for (size_t pi = 0; pi < pools.size(); ++pi) {
        for (int tall = 0; tall < 2; ++tall) {
            std::vector<const Item*> its;
            for (const Item& it : items)
                if (it.pool == (int)pi && (int)it.d.tall == tall &&
                    (!it.gns || iter == 0 || iter == kGnsRestart)) {
                    its.push_back(&it);
                    if ((int)its.size() == kMaxGramGroups) {
                        if (int rc = gram_pool_launch(sc, its, pools[pi], iter, first_it)) return rc;
                        its.clear();
                    }
                }
            if (!its.empty())
                if (int rc = gram_pool_launch(sc, its, pools[pi], iter, first_it)) return rc;
        }
    }
    return NORMPRE_OK;
}

// B = b A + c A^2 for the pool's slots [first, first + cnt) in one launch,
// written to `out` (slot `first` at out[0]).
int poly_launch(const StepCtx& sc, const Pool& pl, int first, int cnt, half_t* out, double nominal_flops) {
    const int64_t sp = pl.sp, ss = sp * sp;
    const half_t* a0 = pl.amat + (int64_t)first * ss;
    Operand A{a0, sp, ss}, B{a0, sp, ss};
    GemmShape sh{(int)sp, (int)sp, (int)sp, 1, (int)sp, 1};
    EpiAffine e{};
    e.out = out; e.ld_out = sp; e.stride_out = ss;
    e.src = a0; e.ld_src = sp; e.stride_src = ss;
    e.ca = sc.hp->ns_coeffs[2]; e.cs = sc.hp->ns_coeffs[1];
    const TileCfg cfg = ns_cfg(sp, sp, sp, true, cnt);
    // Nominal FLOPs use the real s of each matrix (padding excluded); bytes
    // are A read once and B written once (4 s^2 per matrix).
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NS_POLY, nominal_flops, 2.0 * nominal_flops / (double)sp,
                 [&] { return launch_gemm_affine(cfg, 0, A, B, sh, cnt, e, sc.s); },
                 issued_flops(cfg, sp, sp, sp, true, cnt)),
           "ns poly");
    return NORMPRE_OK;
}

// X <- cs X + S X (wide) or X <- cs X + X S (tall) with S the item's slots of
// the pool's s x s matrices `smat` (B for the plain iteration, Q at a
// Gram-space segment end with cs = 0).
int combine_launch(const StepCtx& sc, const Item& it, const half_t* smat, half_t* x, half_t* xn, bool first_it,
                   bool last_it, float cs) {
    const Dims& d = it.d;
    const int count = it.count;
    const int64_t mn = d.mp * d.np_, ss = d.sp * d.sp;
    const double s_ = (double)std::min(d.m, d.n), l_ = (double)std::max(d.m, d.n);
    const half_t* bmat = smat + (int64_t)it.pool_off * ss;
    EpiAffine e{};
    e.out = xn; e.ld_out = d.np_; e.stride_out = mn;
    e.src = cs != 0.f ? x : nullptr; e.ld_src = d.np_; e.stride_src = mn;
    e.mul = first_it ? it.w.scale : nullptr; e.mul_pow = first_it ? 1 : 0;
    e.ca = 1.f; e.cs = cs;
    const TileCfg cfg = it.ccfg;
    e.sumsq = last_it ? it.w.sumsq : nullptr;
    e.tiles_per_mat = combine_tiles(d, cfg);
    auto go = [&]() -> hipError_t {
        if (!d.tall) {
            // X <- a X + B X
            Operand A{bmat, d.sp, ss}, B{x, d.np_, mn};
            GemmShape sh{(int)d.sp, (int)d.lp_, (int)d.sp, 1, (int)d.sp, 0};
            return launch_gemm_affine(cfg, 1, A, B, sh, count, e, sc.s);
        }
        // Y <- a Y + Y B
        Operand A{x, d.np_, mn}, B{bmat, d.sp, ss};
        GemmShape sh{(int)d.lp_, (int)d.sp, (int)d.sp, 1, (int)d.sp, 0};
        return launch_gemm_affine(cfg, 0, A, B, sh, count, e, sc.s);
    };
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NS_COMBINE, 2.0 * s_ * s_ * l_ * count, 2.0 * (2.0 * s_ * l_ + s_ * s_) * count,
                 go, issued_flops(cfg, d.sp, d.lp_, d.sp, false, count)),
           "ns combine");
    return NORMPRE_OK;
}

// The combines of the wide items (m <= n) of one pool, in chunks of up to
// kMaxItems: one launch each, one tile for the chunk from its total tile
// count (ns_cfg's rule), so small shape groups fill the chip together.
std::vector<std::vector<Item*>> wide_combine_chunks(std::vector<Item>& items, size_t npools) {
    std::vector<std::vector<Item*>> chunks;
    for (size_t pi = 0; pi < npools; ++pi) {
        std::vector<Item*> cur;
        for (Item& it : items) {
            if (it.pool != (int)pi || it.d.tall || it.gns) continue;
            cur.push_back(&it);
            if ((int)cur.size() == kMaxItems) {
                chunks.push_back(cur);
                cur.clear();
            }
        }
        if (!cur.empty()) chunks.push_back(cur);
    }
    for (auto& ch : chunks) {
        int64_t tiles = 0;
        for (const Item* it : ch) tiles += (it->d.mp / 256) * (it->d.np_ / 256) * it->count;
        const TileCfg cfg = tiles >= 384 ? TileCfg::Big256 : TileCfg::Big;
        for (Item* it : ch) it->ccfg = cfg;
    }
    return chunks;
}

int combine_grouped_launch(const StepCtx& sc, const std::vector<Item*>& ch, const Pool& pl, int iter, bool first_it,
                           bool last_it) {
    CombineGroups g{};
    int total = 0;
    double flops = 0.0, bytes = 0.0;
    const TileCfg cfg = ch[0]->ccfg;
    const int64_t sp = ch[0]->d.sp;
    for (const Item* it : ch) {
        const Dims& d = it->d;
        const int64_t mn = d.mp * d.np_, ss = d.sp * d.sp;
        if (d.sp != sp || it->ccfg != cfg || d.tall)
            return set_err(sc.ctx, NORMPRE_ERR_HIP, "internal: combines of one launch differ in s or tile");
        half_t* x = (iter & 1) ? it->w.xb : it->w.psi;
        half_t* xn = (iter & 1) ? it->w.psi : it->w.xb;
        const int i = g.n++;
        g.zbeg[i] = total;
        g.a[i] = pl.bmat + (int64_t)it->pool_off * ss; g.lda[i] = d.sp; g.a_stride[i] = ss;
        g.b[i] = x; g.ldb[i] = d.np_; g.b_stride[i] = mn;
        g.N[i] = (int)d.lp_;
        g.out[i] = xn; g.ld_out[i] = d.np_; g.stride_out[i] = mn;
        g.src[i] = x; g.ld_src[i] = d.np_; g.stride_src[i] = mn;
        g.mul[i] = first_it ? it->w.scale : nullptr;
        g.sumsq[i] = last_it ? it->w.sumsq : nullptr;
        g.tiles[i] = combine_tiles(d, cfg);
        const double s_ = (double)std::min(d.m, d.n), l_ = (double)std::max(d.m, d.n);
        flops += 2.0 * s_ * s_ * l_ * it->count;
        bytes += 2.0 * (2.0 * s_ * l_ + s_ * s_) * it->count;
        total += it->count;
    }
    g.zbeg[g.n] = total;
    EpiAffine e{};
    e.mul_pow = first_it ? 1 : 0;
    e.ca = 1.f;
    e.cs = sc.hp->ns_coeffs[0];
    double issued = 0.0;
    for (const Item* it : ch) issued += issued_flops(cfg, sp, it->d.lp_, sp, false, it->count);
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NS_COMBINE, flops, bytes,
                 [&] { return launch_gemm_combine_grouped(cfg, (int)sp, g, e, sc.s); }, issued),
           "ns combine");
    return NORMPRE_OK;
}

// out = S R + cs R for the pool's Gram-space slots (symmetric results: S and R
// are polynomials in the same A_0, so only upper tiles are computed).
int gns_product(const StepCtx& sc, const Pool& pl, const half_t* smat, const half_t* r, half_t* out, float cs,
                double flops) {
    const int64_t sp = pl.sp, ss = sp * sp;
    Operand A{smat, sp, ss}, B{r, sp, ss};
    GemmShape sh{(int)sp, (int)sp, (int)sp, 1, (int)sp, 1};
    EpiAffine e{};
    e.out = out; e.ld_out = sp; e.stride_out = ss;
    e.src = r; e.ld_src = sp; e.stride_src = ss;
    e.ca = 1.f; e.cs = cs;
    const TileCfg cfg = ns_cfg(sp, sp, sp, true, pl.gns_count);
    // Bytes: S and R read once, the result written once (6 s^2 per matrix).
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_NS_POLY, flops, 3.0 * flops / (double)sp,
                 [&] { return launch_gemm_affine(cfg, 0, A, B, sh, pl.gns_count, e, sc.s); },
                 issued_flops(cfg, sp, sp, sp, true, pl.gns_count)),
           "ns gram-space product");
    return NORMPRE_OK;
}

// One Gram-space iteration of a pool's Gram-space items, after the pool's
// B_k = b A_k + c A_k^2 (written into Q's first buffer at a segment start,
// else into the pool's B): Q_{k+1} = P_k at a segment start (a I added in
// place), else a Q_k + B_k Q_k; then either A_{k+1} = P_k (P_k A_k) or, at a
// segment end, the items' X = Q X_base (X_0 in psi -> xb, then X_3 in xb ->
// T in psi).
int gns_iteration(const StepCtx& sc, const std::vector<Item>& items, Pool& pl, int pi, int iter, int q,
                  bool fold_scale) {
    const float a = sc.hp->ns_coeffs[0];
    const bool seg_start = iter == 0 || iter == kGnsRestart;
    const bool seg_end = iter == kGnsRestart - 1 || iter == q - 1;
    double flops = 0.0;
    for (const Item& it : items)
        if (it.pool == pi && it.gns) {
            const double s_ = (double)std::min(it.d.m, it.d.n);
            flops += 2.0 * s_ * s_ * s_ * it.count;
        }
    if (seg_start) {
        pl.qcur = 0;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 4.0 * (double)pl.gns_count * pl.sp,
                     [&] { return launch_add_diag(pl.qmat[0], pl.sp, pl.gns_count, a, sc.s); }),
               "ns gram-space identity");
    } else {
        if (int rc = gns_product(sc, pl, pl.bmat, pl.qmat[pl.qcur], pl.qmat[1 - pl.qcur], a, flops)) return rc;
        pl.qcur = 1 - pl.qcur;
    }
    if (!seg_end) {
        // P_k is Q's first buffer at a segment start (no src term), else B_k + a I.
        const half_t* left = seg_start ? pl.qmat[0] : pl.bmat;
        const float cs = seg_start ? 0.f : a;
        if (int rc = gns_product(sc, pl, left, pl.amat, pl.rmat, cs, flops)) return rc;
        return gns_product(sc, pl, left, pl.rmat, pl.amat, cs, flops);
    }
    const bool first_seg = iter < kGnsRestart;
    for (const Item& it : items) {
        if (it.pool != pi || !it.gns) continue;
        half_t* x = first_seg ? it.w.psi : it.w.xb;
        half_t* xn = first_seg ? it.w.xb : it.w.psi;
        if (int rc = combine_launch(sc, it, pl.qmat[pl.qcur], x, xn, first_seg && fold_scale, iter == q - 1, 0.f))
            return rc;
    }
    return NORMPRE_OK;
}

int g_update_launch(const StepCtx& sc, const Item& it, const half_t* t, DebugMat* dbg) {
    const Dims& d = it.d;
    const normpre_hparams& hp = *sc.hp;
    const std::vector<int>& idx = (*sc.groups)[it.g].idx;
    const int first = it.first, count = it.count;
    const int64_t mn = d.mp * d.np_;
    // ||T||_F^2: NormPre-G from the last combine's per-tile sums; normalize-only
    // (T = Psi) from the normalization's row sums; Muon uses a fixed scale.
    const float* tn2 = it.w.tn2;
    int64_t tn2_stride = 1;
    float fixed_scale = 0.f;
    if (sc.variant == NORMPRE_VARIANT_G) {
        const int t_tiles = combine_tiles(d, it.ccfg);
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                     [&] { return launch_sum_partials(it.w.sumsq, t_tiles, it.w.tn2, count, sc.s); }),
               "t norm");
    } else if (sc.variant == NORMPRE_VARIANT_NORMALIZE_ONLY) {
        tn2 = it.w.scale + 1;
        tn2_stride = 2;
    } else {
        fixed_scale = hp.target_rms * std::sqrt((float)std::max(d.m, d.n));
    }
    for (int c0 = 0; c0 < count; c0 += kChunk) {
        const int cnt = std::min(kChunk, count - c0);
        GUpdateArgs a{};
        a.ptrs = make_chunk(sc, idx, first + c0, cnt);
        a.rows = (int)d.m;
        a.cols = (int)d.n;
        a.t = t + (int64_t)c0 * mn;
        a.ld_t = d.np_;
        a.stride_t = mn;
        a.tnorm2 = tn2 + c0 * tn2_stride;
        a.tnorm2_stride = tn2_stride;
        a.fixed_scale = fixed_scale;
        a.lr = hp.lr;
        a.wd = hp.weight_decay;
        a.target_rms = hp.target_rms;
        a.vec_ok = chunk_vec_ok(a.ptrs, cnt);
        if (dbg) {
            for (int i = 0; i < cnt; ++i) {
                NP_TRY(hipMemcpyAsync(dbg[idx[first + c0 + i]].scalars, tn2 + (c0 + i) * tn2_stride, sizeof(float),
                                      hipMemcpyDeviceToDevice, sc.s),
                       "dbg");
                // one matrix per launch keeps the debug pointers simple
                GUpdateArgs b = a;
                PtrChunk pc{};
                pc.w[0] = a.ptrs.w[i];
                pc.m[0] = a.ptrs.m[i];
                pc.g[0] = a.ptrs.g[i];
                b.ptrs = pc;
                b.t = a.t + (int64_t)i * mn;
                b.tnorm2 = a.tnorm2 + i * tn2_stride;
                b.t32 = dbg[idx[first + c0 + i]].t32;
                b.stride_t32 = d.m * d.n;
                NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_G_UPDATE, 0.0, 10.0 * d.m * d.n,
                             [&] { return launch_g_update(b, 1, sc.s); }),
                       "g update");
            }
            continue;
        }
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_G_UPDATE, 0.0, 10.0 * d.m * d.n * cnt,
                     [&] { return launch_g_update(a, cnt, sc.s); }),
               "g update");
    }
    return NORMPRE_OK;
}

// NormPre-G, and the Muon and normalize-only reference steps, which share
// its stages: input (normalize, or Muon's momentum + Frobenius scaling),
// q Newton-Schulz iterations (none for normalize-only), update.
int run_round_g(const StepCtx& sc, std::vector<Item>& items, std::vector<Pool>& pools, DebugMat* dbg) {
    for (const Item& it : items) {
        int rc = sc.variant == NORMPRE_VARIANT_MUON
                     ? run_muon_input(sc, it.d, it.w, (*sc.groups)[it.g].idx, it.first, it.count, dbg)
                     : run_normalize(sc, it.d, it.w, (*sc.groups)[it.g].idx, it.first, it.count, dbg);
        if (rc) return rc;
    }
    // Muon's X0 is scaled when it is written; NormPre-G folds 1/||Psi||_F
    // into the first iteration's epilogues.
    const bool fold_scale = sc.variant == NORMPRE_VARIANT_G;
    const int q = sc.variant == NORMPRE_VARIANT_NORMALIZE_ONLY ? 0 : sc.hp->ns_iters;
    // Combine tiles: the plain-iteration wide items of a pool share launches;
    // tall and Gram-space items run per item.
    for (Item& it : items)
        if (it.d.tall || it.gns) it.ccfg = ns_cfg(it.d.mp, it.d.np_, it.d.sp, false, it.count);
    const auto wide = wide_combine_chunks(items, pools.size());
    for (int iter = 0; iter < q; ++iter) {
        const bool first_it = iter == 0 && fold_scale, last_it = iter == q - 1;
        int rc = gram_launches(sc, items, pools, iter, first_it);
        if (rc) return rc;
        for (size_t pi = 0; pi < pools.size(); ++pi) {
            Pool& pl = pools[pi];
            double fg = 0.0, fs = 0.0;
            for (const Item& it : items)
                if (it.pool == (int)pi) {
                    const double s_ = (double)std::min(it.d.m, it.d.n);
                    (it.gns ? fg : fs) += 2.0 * s_ * s_ * s_ * it.count;
                }
            // At a Gram-space segment start the Gram-space slots' B goes
            // straight into Q's first buffer (Q_{k+1} = B_k + a I).
            const bool split = pl.gns_count > 0 && (iter == 0 || iter == kGnsRestart);
            int rc = split ? poly_launch(sc, pl, 0, pl.gns_count, pl.qmat[0], fg)
                           : poly_launch(sc, pl, 0, pl.count, pl.bmat, fg + fs);
            if (!rc && split && pl.count > pl.gns_count)
                rc = poly_launch(sc, pl, pl.gns_count, pl.count - pl.gns_count,
                                 pl.bmat + (int64_t)pl.gns_count * pl.sp * pl.sp, fs);
            if (rc) return rc;
        }
        for (const auto& ch : wide) {
            const Item& it0 = *ch[0];
            half_t* x = (iter & 1) ? it0.w.xb : it0.w.psi;
            half_t* xn = (iter & 1) ? it0.w.psi : it0.w.xb;
            // A lone item takes the plain launch (no table to walk).
            int rc = ch.size() == 1 ? combine_launch(sc, it0, pools[it0.pool].bmat, x, xn, first_it, last_it,
                                                     sc.hp->ns_coeffs[0])
                                    : combine_grouped_launch(sc, ch, pools[it0.pool], iter, first_it, last_it);
            if (rc) return rc;
        }
        for (const Item& it : items) {
            if (!it.d.tall || it.gns) continue;
            half_t* x = (iter & 1) ? it.w.xb : it.w.psi;
            half_t* xn = (iter & 1) ? it.w.psi : it.w.xb;
            int rc = combine_launch(sc, it, pools[it.pool].bmat, x, xn, first_it, last_it, sc.hp->ns_coeffs[0]);
            if (rc) return rc;
        }
        for (size_t pi = 0; pi < pools.size(); ++pi) {
            if (pools[pi].gns_count == 0) continue;
            if (int rc = gns_iteration(sc, items, pools[pi], (int)pi, iter, q, fold_scale)) return rc;
        }
    }
    for (const Item& it : items) {
        // Gram-space items end with T in psi (their second segment writes it).
        const half_t* t = it.gns ? it.w.psi : (q & 1) ? it.w.xb : it.w.psi;
        int rc = g_update_launch(sc, it, t, dbg);
        if (rc) return rc;
    }
    return NORMPRE_OK;
}

// One sketch product over Psi with an l-major fp16 operand V (ell_pad x K):
// out_over_active = true gives (Psi V)^T (ell_pad x a_pad), false gives
// (Psi^T V)^T (ell_pad x b_pad).  Writes fp32 and/or scaled fp16 results.
int sketch_product(const StepCtx& sc, const Dims& d, const GWork& w, int count, const half_t* v16, bool over_active,
                   float* out32, half_t* out16, float scale16, const half_t* src = nullptr) {
    const int64_t mn = d.mp * d.np_, lp = d.ellp, maxpad = d.lp_;
    // PV: out over the rows of the W-layout Psi; PtV: over its columns.
    const bool pv = over_active == (d.k == 0);
    const int64_t n_out = pv ? d.mp : d.np_;
    const int64_t k_len = pv ? d.np_ : d.mp;
    const TileCfg cfg = lp == 128 ? TileCfg::Skinny128 : TileCfg::Skinny64;
    const int bm = gemm_tile_m(cfg), bn = gemm_tile_n(cfg);
    const int64_t tiles = (lp / bm) * (n_out / bn);
    const int splits = pick_splits(tiles, count, k_len);
    const int64_t k_chunk = round_up((k_len + splits - 1) / splits, 64);
    const int real_splits = (int)((k_len + k_chunk - 1) / k_chunk);
    Operand A{v16, k_len, lp * maxpad};
    Operand B{src ? src : w.psi, d.np_, mn};
    GemmShape sh{(int)lp, (int)n_out, (int)k_len, real_splits, (int)k_chunk, 0};
    EpiPartial e{};
    e.out = w.part;
    e.ld_out = n_out;
    e.stride_split = lp * n_out;
    e.stride_mat = (int64_t)kMaxSplits * lp * maxpad;
    const double flops = 2.0 * d.ell * (double)d.m * (double)d.n * count;
    const double bytes = 2.0 * (double)d.m * (double)d.n * count;
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_STREAM, flops, bytes,
                 [&] { return launch_gemm_partial(cfg, pv ? 0 : 1, A, B, sh, count, e, sc.s); }),
           "sketch product");
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                 [&] {
                     return launch_reduce_splits(w.part, real_splits, lp * n_out, (int64_t)kMaxSplits * lp * maxpad,
                                                 (int)lp, n_out, out32, out16, scale16, lp * maxpad, count, sc.s);
                 }),
           "reduce splits");
    return NORMPRE_OK;
}

// One sketch-product stage for the items of a pool run: one grouped split-K
// launch and one grouped split reduction (the per-item arithmetic of
// sketch_product).  `pick` gives an item's l-major operand, outputs, fp16
// scale and source (null: Psi).
struct SkIO {
    const half_t* v16;
    float* out32;
    half_t* out16;
    float scale16;
    const half_t* src;
};

template <class Pick>
int sketch_product_run(const StepCtx& sc, const std::vector<const Item*>& its, bool over_active, Pick pick) {
    SketchGroups g{};
    ReduceGroups r{};
    TileCfg cfg = TileCfg::Skinny64;
    int layout = -1, total = 0, rtotal = 0;
    int64_t lp0 = 0;
    double flops = 0.0, bytes = 0.0;
    // l_pad = 64 takes 512-wide output tiles when every product's output
    // length allows it (half the re-reads of the l-major operand per byte of
    // Psi streamed), else 256-wide ones.
    bool wide = true;
    for (const Item* it : its) {
        const bool pv = over_active == (it->d.k == 0);
        wide = wide && ((pv ? it->d.mp : it->d.np_) % 512 == 0);
    }
    auto tile_of = [&](int64_t lp) {
        return lp == 128 ? TileCfg::Skinny128 : wide ? TileCfg::Skinny64W : TileCfg::Skinny64;
    };
    // The split count comes from the launch's total tile count: every item's
    // split chunks fill the chip together.
    int64_t all_tiles = 0;
    for (const Item* it : its) {
        const Dims& d = it->d;
        const bool pv = over_active == (d.k == 0);
        const TileCfg c = tile_of(d.ellp);
        all_tiles += (d.ellp / gemm_tile_m(c)) * ((pv ? d.mp : d.np_) / gemm_tile_n(c)) * it->count;
    }
    for (const Item* it : its) {
        const Dims& d = it->d;
        const GWork& w = it->w;
        const SkIO io = pick(*it);
        const int64_t mn = d.mp * d.np_, lp = d.ellp, maxpad = d.lp_;
        const bool pv = over_active == (d.k == 0);
        const int64_t n_out = pv ? d.mp : d.np_;
        const int64_t k_len = pv ? d.np_ : d.mp;
        const TileCfg c = tile_of(lp);
        if (layout < 0) {
            cfg = c;
            layout = pv ? 0 : 1;
            lp0 = lp;
        } else if (c != cfg || layout != (pv ? 0 : 1) || lp != lp0) {
            return set_err(sc.ctx, NORMPRE_ERR_HIP, "internal: sketch products of one launch differ in l or side");
        }
        const int splits = pick_splits(all_tiles, 1, k_len);
        const int64_t k_chunk = round_up((k_len + splits - 1) / splits, 64);
        const int real_splits = (int)((k_len + k_chunk - 1) / k_chunk);
        const int i = g.n++;
        g.zbeg[i] = total;
        g.a[i] = io.v16; g.lda[i] = k_len; g.a_stride[i] = lp * maxpad;
        g.b[i] = io.src ? io.src : w.psi; g.ldb[i] = d.np_; g.b_stride[i] = mn;
        g.N[i] = (int)n_out; g.K[i] = (int)k_len; g.k_chunk[i] = (int)k_chunk; g.splits[i] = real_splits;
        g.out[i] = w.part; g.stride_split[i] = lp * n_out; g.stride_mat[i] = (int64_t)kMaxSplits * lp * maxpad;
        g.out32[i] = io.out32; g.out16[i] = io.out16; g.scale16[i] = io.scale16; g.stride_out[i] = lp * maxpad;
        // One split: the product launch writes the outputs itself.
        if (real_splits > 1 && (io.out32 || io.out16)) {
            const int j = r.n++;
            r.zbeg[j] = rtotal;
            r.part[j] = w.part; r.splits[j] = real_splits;
            r.stride_split[j] = lp * n_out; r.stride_mat[j] = (int64_t)kMaxSplits * lp * maxpad;
            r.n4[j] = lp * n_out / 4;
            r.out32[j] = io.out32; r.out16[j] = io.out16; r.scale16[j] = io.scale16; r.stride_out[j] = lp * maxpad;
            rtotal += it->count;
        }
        flops += 2.0 * d.ell * (double)d.m * (double)d.n * it->count;
        bytes += 2.0 * (double)d.m * (double)d.n * it->count;
        total += it->count;
    }
    if (g.n == 0) return NORMPRE_OK;
    g.zbeg[g.n] = total;
    r.zbeg[r.n] = rtotal;
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_STREAM, flops, bytes,
                 [&] { return launch_gemm_partial_grouped(cfg, layout, (int)lp0, g, sc.s); }),
           "sketch product");
    if (r.n > 0)
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0, [&] { return launch_reduce_splits_grouped(r, sc.s); }),
               "reduce splits");
    return NORMPRE_OK;
}

// The items of each pool in pool order, in runs of at most kMaxItems (one
// grouped launch each); their matrices are contiguous in the pool buffers.
std::vector<std::vector<const Item*>> pool_runs(const std::vector<Item>& items, const std::vector<Pool>& pools) {
    std::vector<std::vector<const Item*>> runs;
    for (size_t pi = 0; pi < pools.size(); ++pi) {
        std::vector<const Item*> run;
        for (const Item& it : items) {
            if (it.pool != (int)pi) continue;
            run.push_back(&it);
            if ((int)run.size() == kMaxItems) {
                runs.push_back(run);
                run.clear();
            }
        }
        if (!run.empty()) runs.push_back(run);
    }
    return runs;
}

// fp64 Gram partials of one l-major fp32 matrix per item (chosen by `pick`,
// which returns the item's V and its length) for a run of one pool.
template <class Pick>
int gram64_run(const StepCtx& sc, const std::vector<const Item*>& run, const Pool& pl, Pick pick) {
    const int64_t lp = pl.ellp, off0 = run[0]->pool_off;
    Gram64Items t{};
    t.ell = pl.ell;
    for (const Item* it : run) {
        const int g = t.n++;
        int64_t len = 0;
        t.v[g] = pick(*it, len);
        t.zbeg[g] = it->pool_off - (int)off0;
        t.ld[g] = len;
        t.stride[g] = lp * it->d.lp_;
        t.len[g] = len;
        t.chunk_len[g] = gram_chunk_len(len);
        t.zbeg[g + 1] = t.zbeg[g] + it->count;
    }
    double* out = pl.gpart + off0 * kGramChunks * lp * lp;
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0, [&] { return launch_gram64(t, (int)lp, out, sc.s); }),
           "gram64");
    return NORMPRE_OK;
}

// out = M^T V per item for a run of one pool (M from the pool's l x l
// buffer `mats`); `fill` sets the item's V and outputs.
template <class Fill>
int small_mul_run(const StepCtx& sc, const std::vector<const Item*>& run, const Pool& pl, const float* mats,
                  Fill fill, const char* what) {
    const int64_t lp = pl.ellp, off0 = run[0]->pool_off;
    SmallMulArgs a{};
    a.ell = pl.ell;
    a.ell_pad = (int)lp;
    for (const Item* it : run) {
        const int g = a.n++;
        SmallMulItem& m = a.it[g];
        m.mat = mats + (int64_t)it->pool_off * lp * lp;
        fill(*it, m);
        a.zbeg[g] = it->pool_off - (int)off0;
        a.zbeg[g + 1] = a.zbeg[g] + it->count;
    }
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0, [&] { return launch_small_mul(a, sc.s); }), what);
    return NORMPRE_OK;
}

// One Cholesky-QR pass over every item of the round: Gram (one launch per
// pool), Cholesky and inverse (one launch per pool), then Q = Y R^-1 (one
// launch per pool).
int cholqr_round(const StepCtx& sc, std::vector<Item>& items, std::vector<Pool>& pools, bool final_pass) {
    const auto runs = pool_runs(items, pools);
    for (const auto& run : runs) {
        int rc = gram64_run(sc, run, pools[run[0]->pool], [&](const Item& it, int64_t& len) -> const float* {
            len = it.d.a_pad;
            return final_pass ? it.w.v32[1] : it.w.v32[0];
        });
        if (rc) return rc;
    }
    for (const Pool& pl : pools)
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                     [&] {
                         return launch_chol_inv(pl.gpart, kGramChunks, pl.ell, pl.ellp, pl.chol, pl.rinv, pl.count,
                                                sc.s);
                     }),
               "cholesky");
    for (const auto& run : runs) {
        const Pool& pl = pools[run[0]->pool];
        int rc = small_mul_run(
            sc, run, pl, pl.rinv,
            [&](const Item& it, SmallMulItem& m) {
                const int64_t lp = it.d.ellp, maxpad = it.d.lp_, len = it.d.a_pad;
                m.v = final_pass ? it.w.v32[1] : it.w.v32[0];
                m.ld_v = len;
                m.stride_v = lp * maxpad;
                m.len = len;
                m.len_pad = len;
                if (final_pass) {
                    m.out16 = it.w.v16[0]; m.stride_out16 = lp * maxpad;
                    m.out16t = it.w.qlen; m.stride_out16t = len * lp;
                } else {
                    m.out32 = it.w.v32[1]; m.stride_out32 = lp * maxpad;
                }
            },
            "q = y r^-1");
        if (rc) return rc;
    }
    return NORMPRE_OK;
}

float pow2_at_most_inv_sqrt(int64_t a) {
    // 2^-ceil(log2(sqrt(a))): bounds the growth of one product with Psi.
    int e = 0;
    while ((int64_t(1) << (2 * e)) < a) ++e;
    return std::ldexp(1.f, -e);
}

int sketch_front(const StepCtx& sc, const Item& it, DebugMat* dbg) {
    const Dims& d = it.d;
    const GWork& w = it.w;
    const std::vector<int>& idx = (*sc.groups)[it.g].idx;
    const int first = it.first, count = it.count;
    int rc = run_normalize(sc, d, w, idx, first, count, dbg);
    if (rc) return rc;
    const normpre_hparams& hp = *sc.hp;
    const int64_t lp = d.ellp, maxpad = d.lp_;
    // Omega^T (ell_pad x b_pad), one counter per matrix: its index in the list.
    for (int c0 = 0; c0 < count; c0 += kChunk) {
        const int cnt = std::min(kChunk, count - c0);
        OmegaArgs o{};
        o.seed = hp.seed;
        o.step = hp.step;
        for (int i = 0; i < cnt; ++i) o.ids[i] = idx[first + c0 + i];
        o.b = (int)d.b;
        o.ell = d.ell;
        o.ell_pad = (int)lp;
        o.ld = d.b_pad;
        o.out = w.omega + (int64_t)c0 * lp * maxpad;
        o.stride = lp * maxpad;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0, [&] { return launch_omega_f16(o, cnt, sc.s); }),
               "omega");
    }
    return NORMPRE_OK;
}

// Alg. 2: Y = Psi Omega; p times Y <- Psi (Psi^T Y), each product one grouped
// launch over the sketched items of a pool run.  The fp16 copies of Z and Y
// are scaled by powers of two (lambda_max <= tr Gamma <= a bounds each
// product), which only rescales the spanned subspace.  The candidate
// subspace comes from the interaction source: Psi, or the trace-matched X
// (NORMPRE_FLAG_SOURCE_X).
int sketch_power_run(const StepCtx& sc, const std::vector<const Item*>& its) {
    const normpre_hparams& hp = *sc.hp;
    const int p = power_iterations(hp);
    // lambda_max(Gamma) <= tr Gamma = ||Psi||_F^2 <= a (n with both axes).
    auto step_scale = [&](const Item& it) {
        return pow2_at_most_inv_sqrt(hp.orientation == NORMPRE_ORIENT_BOTH ? std::max(it.d.a, it.d.n) : it.d.a);
    };
    int rc = sketch_product_run(sc, its, true, [&](const Item& it) {
        return SkIO{it.w.omega, it.w.v32[0], p > 0 ? it.w.v16[0] : nullptr, 1.f, it.w.xs};
    });
    if (rc) return rc;
    for (int i = 0; i < p; ++i) {
        rc = sketch_product_run(sc, its, false, [&](const Item& it) {
            return SkIO{it.w.v16[0], nullptr, it.w.v16[1], step_scale(it), it.w.xs};
        });
        if (rc) return rc;
        rc = sketch_product_run(sc, its, true, [&](const Item& it) {
            return SkIO{it.w.v16[1], it.w.v32[0], i + 1 < p ? it.w.v16[0] : nullptr, step_scale(it), it.w.xs};
        });
        if (rc) return rc;
    }
    return NORMPRE_OK;
}

// Exact NormPre-L above kMaxEll active rows (App. B, exact eigenspace
// extraction): Gamma = Psi Psi^T of the active side (fp16 MFMA, fp32), its
// leading ell = min(r, a) eigenvectors by the fp64 dense eigensolver, written
// as Y^T in place of the sketch; the common tail (orthonormalization,
// Rayleigh-Ritz, selection of lambda > 1, apply) then works on exactly the
// modes C can come from.
int exact_front(const StepCtx& sc, const Item& it, DebugMat* dbg) {
    const Dims& d = it.d;
    const GWork& w = it.w;
    const std::vector<int>& idx = (*sc.groups)[it.g].idx;
    const int count = it.count;
    int rc = run_normalize(sc, d, w, idx, it.first, count, dbg);
    if (rc) return rc;
    const half_t* src = w.xs ? w.xs : w.psi;
    const int64_t mn = d.mp * d.np_, ap = d.a_pad, a = d.a;
    {
        Operand A{src, d.np_, mn}, B{src, d.np_, mn};
        GemmShape sh{(int)ap, (int)ap, (int)d.b_pad, 1, (int)d.b_pad, 0};
        EpiPartial e{};
        e.out = w.gam32;
        e.ld_out = ap;
        e.stride_split = 0;
        e.stride_mat = ap * ap;
        const double flops = 2.0 * (double)ap * (double)ap * (double)d.b_pad * count;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_STREAM, flops, 2.0 * (double)d.m * (double)d.n * count,
                     [&] { return launch_gemm_gram_f32(d.k == 0 ? 0 : 2, A, B, sh, count, e, sc.s); }),
               "exact gamma");
    }
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_EIGEN, 0.0, 0.0,
                 [&] { return launch_gamma_sym(w.gam32, ap, ap * ap, (int)a, w.tw.A, count, sc.s); }),
           "exact gamma");
    // Algorithmic bytes of the reduction: step j reads and writes the
    // (a - j - 1)^2 trailing fp32 block once.
    const double tri_bytes = 8.0 * ((double)(a - 1) * a * (2 * a - 1) / 6.0) * count;
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_EIGEN, 0.0, tri_bytes,
                 [&] { return launch_tridiagonalize(w.tw, (int)a, count, sc.s); }),
           "tridiagonalize");
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_EIGEN, 0.0, 0.0,
                 [&] { return launch_tri_eigvals(w.tw, (int)a, 0, d.ell, w.lam, d.ell, count, sc.s); }),
           "bisection");
    const int64_t lp = d.ellp, maxpad = d.lp_;
    NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_EIGEN, 0.0, 0.0,
                 [&] {
                     return launch_tri_eigvecs(w.tw, (int)a, w.lam, d.ell, w.v32[0], ap, (int)lp, lp * maxpad, count,
                                               sc.s);
                 }),
           "eigenvectors");
    return NORMPRE_OK;
}

// NormPre-L items whose ||T||_F^2 may come in closed form: the Ritz values
// are those of Psi itself (not with the interaction source X, not the dense
// eigensolver's exact variant).
bool closed_norm(const Item& it) { return !it.d.xl && !it.w.xs; }

// The closed-form ||T||_F^2 of every such item of the round, kMaxItems shape
// groups per launch (see LNormGroups).
int closed_norm_launches(const StepCtx& sc, const std::vector<Item>& items, const std::vector<Pool>& pools) {
    LNormGroups g{};
    g.frac = kClosedNormFrac;
    int total = 0;
    auto flush = [&]() -> int {
        if (g.n == 0) return NORMPRE_OK;
        g.zbeg[g.n] = total;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0, [&] { return launch_l_norm_closed(g, sc.s); }),
               "t norm (closed form)");
        g.n = 0;
        total = 0;
        return NORMPRE_OK;
    };
    for (const Item& it : items) {
        if (!closed_norm(it)) continue;
        const Pool& pl = pools[it.pool];
        const int i = g.n++;
        g.zbeg[i] = total;
        g.psi2[i] = it.w.scale + 1;
        g.ritz[i] = pl.ritz + (int64_t)it.pool_off * pl.top;
        g.ritz_stride[i] = pl.top;
        g.nsel[i] = pl.nsel + it.pool_off;
        g.tn2[i] = it.w.tn2;
        g.need[i] = it.w.lneed;
        total += it.count;
        if (g.n == kMaxItems)
            if (int rc = flush()) return rc;
    }
    return flush();
}

int sketch_back(const StepCtx& sc, const Item& it, const Pool& pl, DebugMat* dbg) {
    const Dims& d = it.d;
    const GWork& w = it.w;
    const std::vector<int>& idx = (*sc.groups)[it.g].idx;
    const int first = it.first, count = it.count;
    const normpre_hparams& hp = *sc.hp;
    const int64_t lp = d.ellp, mn = d.mp * d.np_;
    // T = Psi + L R^T in the W layout, fused with the RMS-matched update.
    const half_t* L = d.k == 0 ? w.qlen : w.flen;
    const half_t* R = d.k == 0 ? w.flen : w.qlen;
    const int64_t l_stride = (d.k == 0 ? d.a_pad : d.b_pad) * lp;
    const int64_t r_stride = (d.k == 0 ? d.b_pad : d.a_pad) * lp;
    // ||T||_F^2: in closed form, ||Psi||_F^2 - sum_C (lambda_i - 1), where the
    // selected modes hold at most a quarter of ||Psi||_F^2; there its error
    // is a few 1e-4 of ||T||^2 (fp16 Q and B) while a norm pass over T would
    // stream Psi once more.  Where they hold more, the subtraction cancels,
    // and those matrices take the norm pass: the same product as the update,
    // reduced to per-tile sums of T^2.  (The closed form needs the Ritz
    // values of Psi itself: not with the interaction source X, nor for the
    // dense eigensolver's exact variant.)
    // (closed_norm_launches ran the closed form for these matrices.)
    const bool closed = closed_norm(it);
    {
        Operand A{L, lp, l_stride};
        Operand B{R, lp, r_stride};
        GemmShape sh{(int)d.mp, (int)d.np_, (int)lp, 1, (int)lp, 0};
        EpiApplyNorm e{};
        e.psi = w.psi; e.ld_psi = d.np_; e.stride_psi = mn;
        e.rows = (int)d.m; e.cols = (int)d.n;
        e.sumsq = w.sumsq; e.tiles_per_mat = apply_tiles(d);
        e.need = closed ? w.lneed : nullptr;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_L_APPLY, 2.0 * d.ell * (double)d.m * d.n * count, 2.0 * d.m * d.n * count,
                     [&] { return launch_gemm_apply_norm(A, B, sh, count, e, sc.s); }),
               "apply norm");
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                     [&] {
                         return launch_sum_partials(w.sumsq, apply_tiles(d), w.tn2, count, sc.s,
                                                    closed ? w.lneed : nullptr);
                     }),
               "t norm");
    }
    for (int c0 = 0; c0 < count; c0 += kChunk) {
        const int cnt = std::min(kChunk, count - c0);
        Operand A{L + (int64_t)c0 * l_stride, lp, l_stride};
        Operand B{R + (int64_t)c0 * r_stride, lp, r_stride};
        GemmShape sh{(int)d.mp, (int)d.np_, (int)lp, 1, (int)lp, 0};
        EpiApplyUpdate e{};
        e.psi = w.psi + (int64_t)c0 * mn; e.ld_psi = d.np_; e.stride_psi = mn;
        e.tnorm2 = w.tn2 + c0;
        e.rows = (int)d.m; e.cols = (int)d.n;
        e.lr = hp.lr; e.wd = hp.weight_decay; e.target_rms = hp.target_rms;
        e.ptrs = make_chunk(sc, idx, first + c0, cnt);
        e.vec_ok = (d.n % 4 == 0) && chunk_vec_ok(e.ptrs, cnt);
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_L_APPLY, 2.0 * d.ell * (double)d.m * d.n * cnt, 10.0 * d.m * d.n * cnt,
                     [&] { return launch_gemm_apply(A, B, sh, cnt, e, sc.s); }),
               "apply");
    }
    if (dbg) {
        for (int i = 0; i < count; ++i) {
            DebugMat& dm = dbg[idx[first + i]];
            const int pz = it.pool_off + i;
            NP_TRY(hipMemcpyAsync(dm.scalars, w.tn2 + i, sizeof(float), hipMemcpyDeviceToDevice, sc.s), "dbg");
            NP_TRY(hipMemcpyAsync(dm.scalars + 1, pl.nsel + pz, sizeof(int), hipMemcpyDeviceToDevice, sc.s), "dbg");
            NP_TRY(hipMemcpyAsync(dm.scalars + 2, pl.ritz + (int64_t)pz * d.top, sizeof(float) * d.top,
                                  hipMemcpyDeviceToDevice, sc.s),
                   "dbg");
        }
    }
    return NORMPRE_OK;
}

int run_round_l(const StepCtx& sc, std::vector<Item>& items, std::vector<Pool>& pools, DebugMat* dbg) {
    for (const Item& it : items) {
        int rc = it.d.xl ? exact_front(sc, it, dbg) : sketch_front(sc, it, dbg);
        if (rc) return rc;
    }
    const auto runs = pool_runs(items, pools);
    for (const auto& run : runs) {
        std::vector<const Item*> sketched;
        for (const Item* it : run)
            if (!it->d.xl) sketched.push_back(it);
        if (int rc = sketch_power_run(sc, sketched)) return rc;
    }
    // Q = qr(Y) by two Cholesky-QR passes (fp64 Gram and factorization).
    int rc = cholqr_round(sc, items, pools, false);
    if (rc) return rc;
    rc = cholqr_round(sc, items, pools, true);
    if (rc) return rc;
    // B = Q^T Psi (ell_pad x b_pad) per pool run, Gamma_Q = B B^T per pool
    // (B = Q^T X_s with the interaction source X).
    for (const auto& run : runs) {
        rc = sketch_product_run(sc, run, false, [&](const Item& it) {
            return SkIO{it.w.v16[0], it.w.v32[0], nullptr, 1.f, it.w.xs};
        });
        if (rc) return rc;
    }
    for (const auto& run : runs) {
        rc = gram64_run(sc, run, pools[run[0]->pool], [&](const Item& it, int64_t& len) -> const float* {
            len = it.d.b_pad;
            return it.w.v32[0];
        });
        if (rc) return rc;
    }
    // Ritz pairs and selection, one launch per pool.
    for (const Pool& pl : pools) {
        EigArgs ea{};
        ea.partial = pl.gpart; ea.chunks = kGramChunks;
        ea.ell = pl.ell; ea.ell_pad = pl.ellp; ea.rank = sc.hp->rank;
        ea.scratch = pl.eigs; ea.kmat = pl.kmat;
        ea.ritz = pl.ritz; ea.ritz_stride = pl.top; ea.nsel = pl.nsel;
        ea.max_sweeps = kEigSweeps;
        NP_TRY(timed(sc.ctx, NORMPRE_KCLASS_SK_SMALL, 0.0, 0.0,
                     [&] {
                         return pl.ell > kEigJacobiMax
                                    ? launch_eig_select_dense(ea, pl.tw, pl.lam, pl.zbuf, pl.count, sc.s)
                                    : launch_eig_select(ea, pl.count, sc.s);
                     }),
               "eigensolver");
    }
    // With the interaction source X the preconditioner still acts on Psi:
    // B = Q^T Psi for the apply.
    for (const Item& it : items) {
        if (!it.w.xs) continue;
        rc = sketch_product(sc, it.d, it.w, it.count, it.w.v16[0], false, it.w.v32[0], nullptr, 1.f);
        if (rc) return rc;
    }
    // F = B^T K (b_pad x ell_pad, fp16), one launch per pool.
    for (const auto& run : runs) {
        const Pool& pl = pools[run[0]->pool];
        rc = small_mul_run(
            sc, run, pl, pl.kmat,
            [&](const Item& it, SmallMulItem& m) {
                const int64_t lp = it.d.ellp;
                m.v = it.w.v32[0]; m.ld_v = it.d.b_pad; m.stride_v = lp * it.d.lp_;
                m.len = it.d.b_pad; m.len_pad = it.d.b_pad;
                m.out16t = it.w.flen; m.stride_out16t = it.d.b_pad * lp;
            },
            "f = b^t k");
        if (rc) return rc;
    }
    rc = closed_norm_launches(sc, items, pools);
    if (rc) return rc;
    for (const Item& it : items) {
        rc = sketch_back(sc, it, pools[it.pool], dbg);
        if (rc) return rc;
    }
    return NORMPRE_OK;
}

int ensure_workspace(normpre_ctx* ctx, size_t bytes, hipStream_t s) {
    if (bytes <= ctx->ws_bytes) return NORMPRE_OK;
    if (ctx->ws) {
        if (ctx->have_stream) (void)hipStreamSynchronize(ctx->last_stream);
        (void)hipStreamSynchronize(s);
        (void)hipFree(ctx->ws);
        ctx->ws = nullptr;
        ctx->ws_bytes = 0;
    }
    const size_t want = bytes + bytes / 8;
    hipError_t e = hipMalloc(&ctx->ws, want);
    if (e != hipSuccess) {
        ctx->ws = nullptr;
        (void)hipGetLastError();
        return set_err(ctx, NORMPRE_ERR_OOM, fmt("workspace allocation of %zu bytes failed", want));
    }
    ctx->ws_bytes = want;
    return NORMPRE_OK;
}

int prepare_debug(normpre_ctx* ctx, int num_mats, const int64_t* shapes, int variant, int k,
                  const normpre_hparams& hp, hipStream_t s) {
    size_t need = 0;
    std::vector<size_t> offs(num_mats);
    // per-matrix psi32 buffers are laid out contiguously per shape group so a
    // chunked launch can address them with one stride
    std::map<std::pair<int64_t, int64_t>, std::vector<int>> by_shape;
    for (int i = 0; i < num_mats; ++i) by_shape[{shapes[2 * i], shapes[2 * i + 1]}].push_back(i);
    std::vector<size_t> psi_off(num_mats), t_off(num_mats), sc_off(num_mats);
    for (auto& kv : by_shape) {
        const int64_t mn = kv.first.first * kv.first.second;
        for (int i : kv.second) { psi_off[i] = need; need += (size_t)mn * 4; }
        for (int i : kv.second) { t_off[i] = need; need += (size_t)mn * 4; }
        for (int i : kv.second) { sc_off[i] = need; need += (size_t)(2 + kMaxEll) * 4; }
    }
    if (need > ctx->dbg_bytes) {
        if (ctx->dbg_mem) {
            (void)hipStreamSynchronize(s);
            (void)hipFree(ctx->dbg_mem);
            ctx->dbg_mem = nullptr;
            ctx->dbg_bytes = 0;
        }
        if (hipMalloc(&ctx->dbg_mem, need) != hipSuccess) {
            ctx->dbg_mem = nullptr;
            (void)hipGetLastError();
            return set_err(ctx, NORMPRE_ERR_OOM, "debug buffer allocation failed");
        }
        ctx->dbg_bytes = need;
    }
    ctx->dbg.assign(num_mats, DebugMat{});
    char* base = static_cast<char*>(ctx->dbg_mem);
    for (int i = 0; i < num_mats; ++i) {
        DebugMat& d = ctx->dbg[i];
        d.rows = shapes[2 * i];
        d.cols = shapes[2 * i + 1];
        d.variant = variant;
        d.k = k;
        d.ell = sketch_width(hp, k == 0 ? d.rows : d.cols);
        d.top = std::min(hp.rank, d.ell);
        d.psi32 = reinterpret_cast<float*>(base + psi_off[i]);
        d.t32 = reinterpret_cast<float*>(base + t_off[i]);
        d.scalars = reinterpret_cast<float*>(base + sc_off[i]);
    }
    return NORMPRE_OK;
}

// Detects overlaps between the caller's buffers (W and M are written).
int check_aliasing(normpre_ctx* ctx, int num_mats, float* const* W, const float* const* G, float* const* M,
                   const int64_t* shapes) {
    struct Range {
        uintptr_t lo, hi;
        int mat;
        bool written;
    };
    std::vector<Range> r;
    r.reserve(3 * (size_t)num_mats);
    for (int i = 0; i < num_mats; ++i) {
        if (!W[i] || !G[i] || !M[i]) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("matrix %d has a null pointer", i));
        const uintptr_t bytes = (uintptr_t)(shapes[2 * i] * shapes[2 * i + 1]) * 4u;
        r.push_back({(uintptr_t)W[i], (uintptr_t)W[i] + bytes, i, true});
        r.push_back({(uintptr_t)M[i], (uintptr_t)M[i] + bytes, i, true});
        r.push_back({(uintptr_t)G[i], (uintptr_t)G[i] + bytes, i, false});
    }
    std::sort(r.begin(), r.end(), [](const Range& a, const Range& b) { return a.lo < b.lo; });
    // Sweep: keep the written range reaching furthest and any range reaching furthest.
    uintptr_t max_hi_w = 0, max_hi_any = 0;
    int mat_w = -1, mat_any = -1;
    for (const Range& x : r) {
        if (x.written && x.lo < max_hi_any)
            return set_err(ctx, NORMPRE_ERR_INVALID_ARG,
                           fmt("buffers of matrices %d and %d overlap (a written buffer is shared)", mat_any, x.mat));
        if (!x.written && x.lo < max_hi_w)
            return set_err(ctx, NORMPRE_ERR_INVALID_ARG,
                           fmt("gradient of matrix %d overlaps a written buffer of matrix %d", x.mat, mat_w));
        if (x.hi > max_hi_any) { max_hi_any = x.hi; mat_any = x.mat; }
        if (x.written && x.hi > max_hi_w) { max_hi_w = x.hi; mat_w = x.mat; }
    }
    return NORMPRE_OK;
}

// The launch plan of one step: equal shapes grouped (first-appearance order),
// groups cut into items of at most item_budget workspace bytes, items packed
// into rounds of at most round_budget bytes; `need` is the largest round.
struct Plan {
    int num_mats = 0;
    std::vector<Group> groups;
    std::vector<std::vector<Item>> rounds;
    size_t need = 0;
    size_t one_matrix = 0;   // the largest single-matrix item of the step
};

// Bytes of the per-matrix non-finite counts at the front of the workspace.
size_t status_bytes(int num_mats) { return ((size_t)num_mats * sizeof(long long) + 255) & ~size_t(255); }

Plan plan_step(int variant, int num_mats, const int64_t* shapes, const normpre_hparams& hp, int k,
               size_t item_budget, size_t round_budget) {
    Plan pl;
    pl.num_mats = num_mats;
    const int opts = step_opts(variant, hp);
    {
        std::map<std::pair<int64_t, int64_t>, int> where;
        for (int i = 0; i < num_mats; ++i) {
            auto key = std::make_pair(shapes[2 * i], shapes[2 * i + 1]);
            auto it = where.find(key);
            if (it == where.end()) {
                where[key] = (int)pl.groups.size();
                pl.groups.push_back({key.first, key.second, {i}});
            } else {
                pl.groups[it->second].idx.push_back(i);
            }
        }
    }
    std::vector<Item> all;
    for (size_t g = 0; g < pl.groups.size(); ++g) {
        const Dims d = dims_of(pl.groups[g].m, pl.groups[g].n, k, hp);
        const int cnt = (int)pl.groups[g].idx.size();
        Item one;
        one.g = (int)g;
        one.count = 1;
        one.d = d;
        one.gns = gram_space_ns(variant, d, hp);
        const size_t per = round_bytes({one}, variant, opts);
        pl.one_matrix = std::max(pl.one_matrix, per);
        const int b = (int)std::max<size_t>(1, std::min<size_t>((size_t)cnt, item_budget / std::max<size_t>(per, 1)));
        for (int first = 0; first < cnt; first += b) {
            Item it;
            it.g = (int)g;
            it.first = first;
            it.count = std::min(b, cnt - first);
            it.d = d;
            it.gns = one.gns;
            all.push_back(it);
        }
    }
    // Rounds: consecutive items whose phases run interleaved, with their
    // small matrices pooled.
    for (const Item& it : all) {
        if (!pl.rounds.empty()) {
            std::vector<Item> trial = pl.rounds.back();
            trial.push_back(it);
            const size_t bytes = round_bytes(trial, variant, opts);
            if (bytes <= round_budget) {
                pl.rounds.back().push_back(it);
                pl.need = std::max(pl.need, bytes);
                continue;
            }
        }
        pl.rounds.push_back({it});
        pl.need = std::max(pl.need, round_bytes(pl.rounds.back(), variant, opts));
    }
    if (opts & kOptCheck) pl.need += status_bytes(num_mats);
    return pl;
}

// Workspace bytes that cover every step of this argument list: both
// orientations under the alternating rule.
size_t workspace_need(int variant, int num_mats, const int64_t* shapes, const normpre_hparams& hp) {
    normpre_hparams h = hp;
    size_t need = 0;
    for (int t = 0; t < 2; ++t) {
        h.step = hp.step + t;
        const int k = step_orientation(variant, h);
        need = std::max(need, plan_step(variant, num_mats, shapes, h, k, kGroupBudget, kRoundBudget).need);
    }
    return need;
}

// Makes stream s wait for the work the context enqueued on another stream
// (the workspace is shared by consecutive steps).
int order_after_last(normpre_ctx* ctx, hipStream_t s) {
    if (!ctx->have_stream || ctx->last_stream == s) return NORMPRE_OK;
    hipError_t e = hipEventRecord(ctx->order_ev, ctx->last_stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, ctx->order_ev, 0);
    if (e != hipSuccess) return hip_fail(ctx, e, "ordering after the previous stream");
    return NORMPRE_OK;
}

// Enqueues every round of a plan on s, with the workspace at ws (ws_bytes).
int run_plan(normpre_ctx* ctx, int variant, Plan& plan, float* const* params, const float* const* grads,
             float* const* momentum, const normpre_hparams* hp, hipStream_t s, void* ws, size_t ws_bytes,
             bool debug) {
    const int opts = step_opts(variant, *hp);
    ctx->dbg_valid = false;
    // Finite check: the per-matrix counts (caller order) at the front of the
    // workspace, the rounds after them.
    long long* status = nullptr;
    size_t front = 0;
    if (opts & kOptCheck) {
        status = static_cast<long long*>(ws);
        front = status_bytes(plan.num_mats);
    }
    ctx->status = status;
    ctx->status_count = status ? plan.num_mats : 0;
    ctx->status_stream = s;
    ctx->timing = (hp->flags & NORMPRE_FLAG_TIME_KERNELS) != 0;
    ctx->stream = s;
    StepCtx sc{ctx, s, hp, params, grads, momentum, variant, debug, &plan.groups, status};
    for (std::vector<Item>& items : plan.rounds) {
        std::vector<Pool> pools = make_pools(items, variant);
        Arena ar{static_cast<char*>(ws) + front, 0, ws_bytes - front};
        carve_round(ar, items, pools, variant, opts);
        if (front + ar.off > ws_bytes) return set_err(ctx, NORMPRE_ERR_HIP, "internal: round exceeds the workspace");
        DebugMat* dbg = debug ? ctx->dbg.data() : nullptr;
        int rc = variant == NORMPRE_VARIANT_L ? run_round_l(sc, items, pools, dbg) : run_round_g(sc, items, pools, dbg);
        if (rc) return rc;
    }
    ctx->last_stream = s;
    ctx->have_stream = true;
    if (debug) {
        ctx->dbg_valid = true;
        ctx->dbg_stream = s;
    }
    return NORMPRE_OK;
}

// Common entry checks of the step entry points; on success *s is the stream.
int step_prologue(normpre_ctx* ctx, int variant, int num_mats, float* const* params, const float* const* grads,
                  float* const* momentum, const int64_t* shapes, const normpre_hparams* hp) {
    Fail f = validate(variant, num_mats, shapes, hp);
    if (f.code) return set_err(ctx, f.code, f.msg);
    if (num_mats == 0) return NORMPRE_OK;
    if (!params || !grads || !momentum) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "pointer array is null");
    int rc = check_aliasing(ctx, num_mats, params, grads, momentum, shapes);
    if (rc) return rc;
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    return NORMPRE_OK;
}

}  // namespace

// =========================================================== C ABI ========
extern "C" {

const char* normpre_version(void) { return "normpre-mi355x 0.1 (gfx950, fp16 MFMA, fp32 accumulate)"; }

int normpre_default_hparams(normpre_hparams* hp) {
    if (!hp) return NORMPRE_ERR_INVALID_ARG;
    std::memset(hp, 0, sizeof *hp);
    hp->lr = 6e-4f;
    hp->momentum = 0.95f;
    hp->weight_decay = 0.1f;
    hp->target_rms = 0.2f;
    hp->ns_iters = 5;
    hp->ns_coeffs[0] = 3.4445f;
    hp->ns_coeffs[1] = -4.7750f;
    hp->ns_coeffs[2] = 2.0315f;
    hp->ns_eps = 1e-7f;
    hp->rank = 32;
    hp->oversample = 8;
    hp->power_iters = 1;
    hp->orientation = NORMPRE_ORIENT_ALTERNATING;
    hp->seed = 1337;
    hp->step = 0;
    hp->norm_eps = 1e-12f;
    hp->flags = 0;
    return NORMPRE_OK;
}

int normpre_init(normpre_ctx** ctx, int device) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "ctx is null");
    *ctx = nullptr;
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || device < 0 || device >= count)
        return set_err(nullptr, NORMPRE_ERR_HIP, fmt("no HIP device %d (%d visible)", device, e == hipSuccess ? count : 0));
    normpre_ctx* c = new (std::nothrow) normpre_ctx();
    if (!c) return set_err(nullptr, NORMPRE_ERR_OOM, "context allocation failed");
    c->device = device;
    int prev = 0;
    (void)hipGetDevice(&prev);
    e = hipSetDevice(device);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->order_ev, hipEventDisableTiming);
    // The static scratch array of normpre_step_noalloc: its address on this
    // device (each device holds its own copy of the array).
    if (e == hipSuccess) e = hipGetSymbolAddress(&c->scratch, HIP_SYMBOL(scratch));
    (void)hipSetDevice(prev);
    if (e != hipSuccess) {
        if (c->order_ev) (void)hipEventDestroy(c->order_ev);
        delete c;
        return set_err(nullptr, NORMPRE_ERR_HIP, fmt("context set-up on device %d: %s", device, hipGetErrorString(e)));
    }
    *ctx = c;
    return NORMPRE_OK;
}

void normpre_destroy(normpre_ctx* ctx) {
    if (!ctx) return;
    int prev = 0;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(ctx->device);
    if (ctx->have_stream) (void)hipStreamSynchronize(ctx->last_stream);
    for (auto& p : ctx->pending) {
        (void)hipEventDestroy(p.start);
        (void)hipEventDestroy(p.stop);
    }
    for (hipEvent_t e : ctx->event_pool) (void)hipEventDestroy(e);
    if (ctx->order_ev) (void)hipEventDestroy(ctx->order_ev);
    if (ctx->ws) (void)hipFree(ctx->ws);
    if (ctx->dbg_mem) (void)hipFree(ctx->dbg_mem);
    (void)hipSetDevice(prev);
    delete ctx;
}

const char* normpre_last_error(const normpre_ctx* ctx) {
    return ctx ? ctx->err.c_str() : g_noctx_error.c_str();
}

int normpre_validate(int variant, int num_mats, const int64_t* shapes, const normpre_hparams* hp, char* msg,
                     int msg_len) {
    Fail f = validate(variant, num_mats, shapes, hp);
    if (msg && msg_len > 0) {
        std::strncpy(msg, f.msg.c_str(), (size_t)msg_len - 1);
        msg[msg_len - 1] = '\0';
    }
    return f.code;
}

int normpre_step(normpre_ctx* ctx, int variant, int num_mats, float* const* params, const float* const* grads,
                 float* const* momentum, const int64_t* shapes, const normpre_hparams* hp, void* stream) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    ctx->err.clear();
    int rc = step_prologue(ctx, variant, num_mats, params, grads, momentum, shapes, hp);
    if (rc || num_mats == 0) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int k = step_orientation(variant, *hp);
    Plan plan = plan_step(variant, num_mats, shapes, *hp, k, kGroupBudget, kRoundBudget);
    if (plan.need > ctx->ws_bytes && ctx->reserved)
        return set_err(ctx, NORMPRE_ERR_UNSUPPORTED,
                       fmt("the step needs %zu workspace bytes, %zu are reserved (normpre_reserve)", plan.need,
                           ctx->ws_bytes));
    rc = ensure_workspace(ctx, plan.need, s);
    if (rc) return rc;
    const bool debug = (hp->flags & NORMPRE_FLAG_DEBUG) != 0;
    if (debug) {
        rc = prepare_debug(ctx, num_mats, shapes, variant, k, *hp, s);
        if (rc) return rc;
    }
    rc = order_after_last(ctx, s);
    if (rc) return rc;
    return run_plan(ctx, variant, plan, params, grads, momentum, hp, s, ctx->ws, ctx->ws_bytes, debug);
}

int normpre_workspace_size(int variant, int num_mats, const int64_t* shapes, const normpre_hparams* hp,
                           int64_t* bytes) {
    if (!bytes) return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "bytes is null");
    *bytes = 0;
    Fail f = validate(variant, num_mats, shapes, hp);
    if (f.code) return set_err(nullptr, f.code, f.msg);
    if (num_mats > 0) *bytes = (int64_t)workspace_need(variant, num_mats, shapes, *hp);
    return NORMPRE_OK;
}

int normpre_reserve(normpre_ctx* ctx, int variant, int num_mats, const int64_t* shapes, const normpre_hparams* hp,
                    void* stream) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    ctx->err.clear();
    Fail f = validate(variant, num_mats, shapes, hp);
    if (f.code) return set_err(ctx, f.code, f.msg);
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const size_t need = num_mats > 0 ? workspace_need(variant, num_mats, shapes, *hp) : 0;
    if (need > ctx->ws_bytes) {
        int rc = ensure_workspace(ctx, need, static_cast<hipStream_t>(stream));
        if (rc) return rc;
    }
    ctx->reserved = true;
    return NORMPRE_OK;
}

int normpre_workspace_bytes(const normpre_ctx* ctx, int64_t* bytes) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    if (!bytes) return NORMPRE_ERR_INVALID_ARG;
    *bytes = (int64_t)ctx->ws_bytes;
    return NORMPRE_OK;
}

int normpre_step_noalloc(normpre_ctx* ctx, int variant, int num_mats, float* const* params,
                         const float* const* grads, float* const* momentum, const int64_t* shapes,
                         const normpre_hparams* hp, void* stream) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    ctx->err.clear();
    if (hp && (hp->flags & (NORMPRE_FLAG_DEBUG | NORMPRE_FLAG_TIME_KERNELS)))
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG,
                       "NORMPRE_FLAG_DEBUG and NORMPRE_FLAG_TIME_KERNELS need allocations; not with normpre_step_noalloc");
    int rc = step_prologue(ctx, variant, num_mats, params, grads, momentum, shapes, hp);
    if (rc || num_mats == 0) return rc;
    if (!ctx->scratch) return set_err(ctx, NORMPRE_ERR_HIP, "the scratch array has no device address");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int k = step_orientation(variant, *hp);
    const size_t front = (hp->flags & NORMPRE_FLAG_CHECK_FINITE) ? status_bytes(num_mats) : 0;
    if (front >= kScratchBytes) return set_err(ctx, NORMPRE_ERR_UNSUPPORTED, "too many matrices for the static scratch");
    Plan plan = plan_step(variant, num_mats, shapes, *hp, k, kScratchBytes - front, kScratchBytes - front);
    if (plan.one_matrix + front > kScratchBytes || plan.need > kScratchBytes)
        return set_err(ctx, NORMPRE_ERR_UNSUPPORTED,
                       fmt("a matrix of this step needs %zu workspace bytes; the static scratch holds %zu",
                           std::max(plan.one_matrix, plan.need), kScratchBytes));
    rc = order_after_last(ctx, s);
    if (rc) return rc;
    return run_plan(ctx, variant, plan, params, grads, momentum, hp, s, ctx->scratch, kScratchBytes, false);
}

int normpre_spectrum(normpre_ctx* ctx, int which, int64_t rows, int64_t cols, const float* w, const float* m,
                     const normpre_hparams* hp, double* eigs, void* stream) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    ctx->err.clear();
    if (which != NORMPRE_SPECTRUM_GAMMA && which != NORMPRE_SPECTRUM_GX)
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("unknown spectrum %d", which));
    if (!w || !m || !eigs || !hp) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "null pointer argument");
    if (hp->orientation == NORMPRE_ORIENT_BOTH)
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "the spectrum needs a single active side");
    // The momentum step is not repeated: M is taken as the update source
    // (a zero previous momentum with M as the "gradient" at mu = 0).
    normpre_hparams h = *hp;
    h.momentum = 0.f;
    h.flags &= NORMPRE_FLAG_TANGENT_NONE | NORMPRE_FLAG_TANGENT_STRICT;
    const int64_t shape[2] = {rows, cols};
    Fail f = validate(NORMPRE_VARIANT_NORMALIZE_ONLY, 1, shape, &h);
    if (f.code) return set_err(ctx, f.code, f.msg);
    const int k = orientation_of(h);
    const Dims d = dims_of(rows, cols, k, h);
    if (d.a > kMaxExactRows)
        return set_err(ctx, NORMPRE_ERR_UNSUPPORTED,
                       fmt("spectrum of %lld active rows exceeds %lld", (long long)d.a, (long long)kMaxExactRows));
    const uintptr_t nbytes = (uintptr_t)(rows * cols) * 4u;
    if ((uintptr_t)w < (uintptr_t)m + nbytes && (uintptr_t)m < (uintptr_t)w + nbytes)
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "W and M overlap");
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool gx = which == NORMPRE_SPECTRUM_GX;
    const int64_t a = d.a, ap = d.a_pad;
    Item it;
    it.count = 1;
    it.d = d;
    auto carve = [&](Arena& ar, float*& mcopy) {
        carve_item(ar, it, NORMPRE_VARIANT_NORMALIZE_ONLY, false);
        GWork& g = it.w;
        if (gx) {
            g.xs = ar.take<half_t>(d.mp * d.np_);
            g.xsq = ar.take<float>(d.lp_);
            g.xtot = ar.take<float>(2);
        }
        g.gam32 = ar.take<float>(ap * ap);
        g.tw.A = ar.take<float>(a * a);
        g.tw.vec = ar.take<double>(4 * a);
        g.tw.d = ar.take<double>(a);
        g.tw.e = ar.take<double>(a);
        g.tw.tau = ar.take<double>(a);
        g.lam = ar.take<double>(a);
        mcopy = ar.take<float>(round_up(rows * cols, 4));   // whole 16-byte blocks for the clear
        return ar.off + 256;
    };
    float* mcopy = nullptr;
    Arena probe{nullptr, 0, 0};
    int rc = ensure_workspace(ctx, carve(probe, mcopy), s);
    if (rc) return rc;
    rc = order_after_last(ctx, s);
    if (rc) return rc;
    Arena ar{static_cast<char*>(ctx->ws), 0, ctx->ws_bytes};
    carve(ar, mcopy);
    ctx->timing = false;
    ctx->stream = s;
    ctx->status = nullptr;
    std::vector<Group> groups{{rows, cols, {0}}};
    float* Wl[1] = {const_cast<float*>(w)};    // read only: the normalization reads W
    const float* Gl[1] = {m};
    float* Ml[1] = {mcopy};
    StepCtx sc{ctx, s, &h, Wl, Gl, Ml, NORMPRE_VARIANT_NORMALIZE_ONLY, false, &groups};
    NP_TRY(launch_fill_zero(mcopy, round_up(rows * cols, 4) * 4, s), "clear momentum copy");
    rc = run_normalize(sc, d, it.w, groups[0].idx, 0, 1, nullptr);
    if (rc) return rc;
    const half_t* src = gx ? it.w.xs : it.w.psi;
    {
        const int64_t mn = d.mp * d.np_;
        Operand A{src, d.np_, mn}, B{src, d.np_, mn};
        GemmShape sh{(int)ap, (int)ap, (int)d.b_pad, 1, (int)d.b_pad, 0};
        EpiPartial ep{};
        ep.out = it.w.gam32;
        ep.ld_out = ap;
        ep.stride_mat = ap * ap;
        NP_TRY(launch_gemm_gram_f32(k == 0 ? 0 : 2, A, B, sh, 1, ep, s), "spectrum gram");
    }
    NP_TRY(launch_gamma_sym(it.w.gam32, ap, ap * ap, (int)a, it.w.tw.A, 1, s), "spectrum gram");
    NP_TRY(launch_tridiagonalize(it.w.tw, (int)a, 1, s), "tridiagonalize");
    NP_TRY(launch_tri_eigvals(it.w.tw, (int)a, 0, (int)a, it.w.lam, a, 1, s), "bisection");
    NP_TRY(hipMemcpyAsync(eigs, it.w.lam, (size_t)a * sizeof(double), hipMemcpyDeviceToHost, s), "copy eigenvalues");
    NP_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
    ctx->last_stream = s;
    ctx->have_stream = true;
    return NORMPRE_OK;
}

int normpre_descent_alignment(normpre_ctx* ctx, int num_mats, const float* const* grads,
                              const float* const* w_before, const float* const* w_after, const int64_t* shapes,
                              float lr, float weight_decay, double* cosines, double* mean, void* stream) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    ctx->err.clear();
    if (num_mats < 0) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "num_mats < 0");
    if (!mean) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "mean is null");
    if (!(lr > 0.f) || !std::isfinite(lr) || !std::isfinite(weight_decay))
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "lr must be finite and > 0, weight_decay finite");
    *mean = 0.0;
    if (num_mats == 0) return NORMPRE_OK;
    if (!grads || !w_before || !w_after || !shapes || !cosines)
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "null pointer argument");
    for (int i = 0; i < num_mats; ++i) {
        if (!grads[i] || !w_before[i] || !w_after[i])
            return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("matrix %d has a null pointer", i));
        if (shapes[2 * i] < 1 || shapes[2 * i + 1] < 1 || shapes[2 * i] > kMaxDim || shapes[2 * i + 1] > kMaxDim)
            return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("matrix %d has a bad shape", i));
    }
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t part_n = (size_t)num_mats * kAlignBlocks * 3;
    const size_t need = (part_n + num_mats + 1) * sizeof(double) + 256;
    int rc = ensure_workspace(ctx, need, s);
    if (rc) return rc;
    rc = order_after_last(ctx, s);
    if (rc) return rc;
    ctx->status = nullptr;
    double* part = static_cast<double*>(ctx->ws);
    double* cos_dev = part + part_n;
    double* mean_dev = cos_dev + num_mats;
    for (int c0 = 0; c0 < num_mats; c0 += kChunk) {
        const int cnt = std::min(kChunk, num_mats - c0);
        AlignChunk ch{};
        for (int i = 0; i < cnt; ++i) {
            ch.g[i] = grads[c0 + i];
            ch.wb[i] = w_before[c0 + i];
            ch.wa[i] = w_after[c0 + i];
            ch.n[i] = shapes[2 * (c0 + i)] * shapes[2 * (c0 + i) + 1];
        }
        e = launch_alignment_partials(ch, cnt, (double)lr, (double)weight_decay,
                                      part + (size_t)c0 * kAlignBlocks * 3, s);
        if (e != hipSuccess) return hip_fail(ctx, e, "alignment partials");
    }
    e = launch_alignment_finalize(part, num_mats, cos_dev, mean_dev, s);
    if (e != hipSuccess) return hip_fail(ctx, e, "alignment finalize");
    e = hipMemcpyAsync(cosines, cos_dev, sizeof(double) * num_mats, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(mean, mean_dev, sizeof(double), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(ctx, e, "alignment copy");
    ctx->last_stream = s;
    ctx->have_stream = true;
    return NORMPRE_OK;
}

int normpre_nonfinite_counts(normpre_ctx* ctx, int64_t* counts, int num_mats) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    if (!counts) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "counts is null");
    if (!ctx->status) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "no step with NORMPRE_FLAG_CHECK_FINITE recorded");
    if (num_mats != ctx->status_count)
        return set_err(ctx, NORMPRE_ERR_INVALID_ARG,
                       fmt("num_mats %d differs from the %d matrices of the checked step", num_mats, ctx->status_count));
    hipError_t e = hipSetDevice(ctx->device);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->status_stream);
    if (e == hipSuccess)
        e = hipMemcpy(counts, ctx->status, sizeof(long long) * (size_t)num_mats, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "non-finite counts");
    return NORMPRE_OK;
}

int normpre_stream_ceiling(int mix, int64_t n, const float* a, const float* b, const float* c, float* out32,
                           void* out16, void* stream) {
    if (mix < 0 || mix > 3 || n < 4 || n % 4 || !a) return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "bad stream probe");
    if ((mix <= 1 && (!b || !c)) || (mix == 2 && !b) || (mix != 2 && !out32) || ((mix == 0 || mix == 2) && !out16))
        return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "null buffer for this mix");
    const void* ptrs[] = {a, b, c, out32, out16};
    for (const void* q : ptrs)
        if (reinterpret_cast<uintptr_t>(q) & 15) return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    hipError_t e = launch_stream_probe(mix, n, a, b, c, out32, static_cast<half_t*>(out16), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return set_err(nullptr, NORMPRE_ERR_HIP, fmt("stream probe: %s", hipGetErrorString(e)));
    return NORMPRE_OK;
}

int normpre_energy_split(const double* eigs, int64_t count, int32_t rank, double* out) {
    if (!eigs || !out || count < 0 || rank < 0)
        return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "null pointer or negative count / rank");
    double top = 0.0, remain = 0.0, sub = 0.0;
    int32_t taken = 0;
    for (int64_t i = 0; i < count; ++i) {
        const double lam = eigs[i];
        if (!(lam > 0.0)) continue;
        const double r = std::sqrt(lam) - 1.0, e = r * r;
        if (lam > 1.0) {
            if (taken < rank) {
                top += e;
                ++taken;
            } else {
                remain += e;
            }
        } else if (lam < 1.0) {
            sub += e;
        }
    }
    out[0] = top;
    out[1] = remain;
    out[2] = sub;
    out[3] = top + remain + sub;
    return NORMPRE_OK;
}

int normpre_debug_fetch(normpre_ctx* ctx, int index, int what, void* host_out, int64_t capacity, int64_t* written) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    if (written) *written = 0;
    if (!ctx->dbg_valid) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "no step with NORMPRE_FLAG_DEBUG recorded");
    if (index < 0 || index >= (int)ctx->dbg.size()) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "index out of range");
    if (!host_out) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "host_out is null");
    const DebugMat& d = ctx->dbg[index];
    const void* src = nullptr;
    int64_t bytes = 0;
    int32_t scalar = 0;
    switch (what) {
        case NORMPRE_DEBUG_PSI: src = d.psi32; bytes = d.rows * d.cols * 4; break;
        case NORMPRE_DEBUG_T:
            if (d.variant == NORMPRE_VARIANT_L) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "T is not kept for NormPre-L");
            src = d.t32; bytes = d.rows * d.cols * 4; break;
        case NORMPRE_DEBUG_RITZ:
            if (d.variant != NORMPRE_VARIANT_L) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "Ritz values are NormPre-L only");
            src = d.scalars + 2; bytes = (int64_t)d.top * 4; break;
        case NORMPRE_DEBUG_NSEL:
            if (d.variant != NORMPRE_VARIANT_L) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "the selection is NormPre-L only");
            src = d.scalars + 1; bytes = 4; break;
        case NORMPRE_DEBUG_ELL:
            if (d.variant != NORMPRE_VARIANT_L) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "the sketch is NormPre-L only");
            scalar = d.ell; bytes = 4; break;
        case NORMPRE_DEBUG_TNORM2: src = d.scalars; bytes = 4; break;
        case NORMPRE_DEBUG_ORIENT: scalar = d.k; bytes = 4; break;
        default: return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("unknown debug item %d", what));
    }
    if (capacity < bytes) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, fmt("capacity %lld < %lld bytes", (long long)capacity, (long long)bytes));
    if (!src) {
        std::memcpy(host_out, &scalar, 4);
    } else {
        hipError_t e = hipSetDevice(ctx->device);
        if (e == hipSuccess) e = hipStreamSynchronize(ctx->dbg_stream);
        if (e == hipSuccess) e = hipMemcpy(host_out, src, (size_t)bytes, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(ctx, e, "debug fetch");
    }
    if (written) *written = bytes;
    return NORMPRE_OK;
}

int normpre_sketch_omega(uint64_t seed, int64_t step, int32_t matrix_id, int64_t b, int32_t l, float* dev_out,
                         void* stream) {
    if (!dev_out || b < 1 || l < 1) return set_err(nullptr, NORMPRE_ERR_INVALID_ARG, "bad omega arguments");
    hipError_t e = launch_omega_f32(seed, step, matrix_id, b, l, dev_out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return set_err(nullptr, NORMPRE_ERR_HIP, fmt("omega launch: %s", hipGetErrorString(e)));
    return NORMPRE_OK;
}

int normpre_kernel_stats(normpre_ctx* ctx, int kclass, int64_t* launches, double* device_ms, double* flops,
                         double* exec_flops, double* bytes, int reset) {
    if (!ctx) return set_err(nullptr, NORMPRE_ERR_NOT_INITIALIZED, "context is null");
    if (kclass < 0 || kclass >= NORMPRE_KCLASS_COUNT) return set_err(ctx, NORMPRE_ERR_INVALID_ARG, "kclass out of range");
    int rc = collect_events(ctx);
    if (rc) return rc;
    const KStat& s = ctx->stats[kclass];
    if (launches) *launches = s.launches;
    if (device_ms) *device_ms = s.ms;
    if (flops) *flops = s.flops;
    if (exec_flops) *exec_flops = s.exec_flops;
    if (bytes) *bytes = s.bytes;
    if (reset) ctx->stats[kclass] = KStat{};
    return NORMPRE_OK;
}

}  // extern "C"
