// Batched fp16 x fp16 -> fp32 MFMA GEMMs for gfx950 (v_mfma_f32_32x32x16_f16).
//
// One kernel template serves every dense contraction of the NormPre step:
//   * the Newton-Schulz products A = X X^T, B = bA + cA^2, X <- aX + BX
//     (NormPre-G, Sec. 3.2; quintic of the Muon iteration),
//   * the sketch products Psi Omega, Psi^T Y, Psi Z, Q^T Psi of Alg. 2
//     (NormPre-L, App. B), split along K with fp32 partials,
//   * the localized apply T = Psi + U_C (Lambda_C^{-1/2} - I) U_C^T Psi
//     fused with the RMS-matched weight update of Alg. 1.
//
// C(mm, nn) = sum_k Aop(mm, k) Bop(nn, k).  Each operand is either K-major
// (op(r, k) = p[r*ld + k]) or MN-major (op(r, k) = p[k*ld + r]).  Both are
// staged into LDS in their memory orientation with 16-byte stores: K-major
// tiles as rows of 64 halves (128 B) with an XOR swizzle of the 16-byte
// chunk index, MN-major tiles as 64 k-rows of R halves, whose fragments the
// transposing LDS read (ds_read_b64_tr_b16) returns K-contiguous.
// All sizes are multiples of the tile sizes (the workspace is zero padded).
#include "np_internal.h"

#include <algorithm>
#include <type_traits>
#include <utility>

#include <hip/hip_ext.h>

namespace np {
namespace {

constexpr int BK = 64;
// Native 16-byte vector (HIP's uint4 is a class type whose copies block
// register promotion of the staging arrays).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_idx(int row, int chunk) {
    return row * BK + ((chunk ^ swz(row)) << 3);
}

// R x 64 K-major tile: each thread moves R*8/NT chunks of 16 bytes.  The
// staging registers are a plain array owned by the kernel (not a member), so
// they stay in VGPRs.
template <int R, int NT>
struct KMajorLoader {
    static constexpr bool kTrans = false;
    static constexpr int N = R * 8 / NT;
    static_assert(N >= 1 && R * 8 % NT == 0, "tile too small for the block");
    static __device__ __forceinline__ void load(u32x4 (&r)[N], const half_t* base, int64_t ld, int row0, int k0,
                                                int tid) {
        const half_t* p = base + (int64_t)(row0 + (tid >> 3)) * ld + k0 + (tid & 7) * 8;
        const int64_t step = (int64_t)(NT / 8) * ld;
#pragma unroll
        for (int i = 0; i < N; ++i) r[i] = *reinterpret_cast<const u32x4*>(p + i * step);
    }
    static __device__ __forceinline__ void store(const u32x4 (&r)[N], half_t* lds, int tid) {
#pragma unroll
        for (int i = 0; i < N; ++i) store_item(r, lds, tid, i);
    }
    // Single items, so the stores and loads of one K-step can be spread over
    // its MFMA sub-steps.
    static __device__ __forceinline__ void load_item(u32x4 (&r)[N], const half_t* base, int64_t ld, int row0, int k0,
                                                     int tid, int i) {
        r[i] = *reinterpret_cast<const u32x4*>(base + (int64_t)(row0 + (tid >> 3) + i * (NT / 8)) * ld + k0 +
                                               (tid & 7) * 8);
    }
    static __device__ __forceinline__ void store_item(const u32x4 (&r)[N], half_t* lds, int tid, int i) {
        const int row = (tid >> 3) + i * (NT / 8), ch = tid & 7;
        *reinterpret_cast<u32x4*>(lds + lds_idx(row, ch)) = r[i];
    }
    // 32 x 16 fragment of the 32x32x16 MFMA: lane l gets row mb + l % 32,
    // k = 16 s + 8 (l / 32) .. + 7.
    static __device__ __forceinline__ f16x8 frag(const half_t* lds, int mb, int s, int lane) {
        return *reinterpret_cast<const f16x8*>(lds + lds_idx(mb + (lane & 31), s * 2 + (lane >> 5)));
    }
};

// 64 x R MN-major tile (k rows, r contiguous), kept in that orientation in
// LDS: row k holds R halves, its 16-byte chunk c stored at c ^ mswz(k), and
// the MFMA fragments are read with ds_read_b64_tr_b16.  Within each 16-lane
// group that instruction returns to lane j the j-th column of the 4 x 16
// block the group addresses (lane p supplies row p / 4, halves 4 (p % 4) ..
// 4 (p % 4) + 3), i.e. four consecutive k of one mn index; two such reads
// make one K-contiguous 8-half fragment.  mswz spreads the four rows one
// group reads over disjoint bank ranges.
template <int R, int NT>
struct MNMajorLoader {
    static constexpr bool kTrans = true;
    static constexpr int CH = R / 8;                 // 16-byte chunks per row
    static constexpr int N = R * BK / 8 / NT;
    static_assert(R >= 128 && N >= 1 && R * BK / 8 % NT == 0 && NT % CH == 0, "unsupported MN-major tile");
    static __device__ __forceinline__ int mswz(int k) { return (4 * (k & 3)) & (CH - 1); }
    static __device__ __forceinline__ void load_item(u32x4 (&r)[N], const half_t* base, int64_t ld, int row0, int k0,
                                                     int tid, int i) {
        // The per-thread part of the address does not depend on the K-step
        // (hoisted out of the loop); k0 * ld is wave-uniform (scalar).
        const int k = tid / CH + i * (NT / CH), c = tid % CH;
        const half_t* p = base + (int64_t)k * ld + row0 + c * 8;
        r[i] = *reinterpret_cast<const u32x4*>(p + (int64_t)k0 * ld);
    }
    static __device__ __forceinline__ void store_item(const u32x4 (&r)[N], half_t* lds, int tid, int i) {
        const int k = tid / CH + i * (NT / CH), c = tid % CH;
        *reinterpret_cast<u32x4*>(lds + k * R + ((c ^ mswz(k)) << 3)) = r[i];
    }
    static __device__ __forceinline__ void load(u32x4 (&r)[N], const half_t* base, int64_t ld, int row0, int k0,
                                                int tid) {
#pragma unroll
        for (int i = 0; i < N; ++i) load_item(r, base, ld, row0, k0, tid, i);
    }
    static __device__ __forceinline__ void store(const u32x4 (&r)[N], half_t* lds, int tid) {
#pragma unroll
        for (int i = 0; i < N; ++i) store_item(r, lds, tid, i);
    }
    // 32 x 16 fragment of the 32x32x16 MFMA: lane l gets mn = mb + l % 32,
    // k = 16 s + 8 (l / 32) .. + 7.
    static __device__ __forceinline__ f16x8 frag(const half_t* lds, int mb, int s, int lane) {
        const int g = lane >> 4, p = lane & 15;
        const int c = (mb >> 3) + 2 * (g & 1) + ((p & 3) >> 1);
        const int k = 16 * s + 8 * (g >> 1) + (p >> 2);
        const int within = 4 * (p & 1);
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
        const half_t* a0 = lds + k * R + ((c ^ mswz(k)) << 3) + within;
        const half_t* a1 = lds + (k + 4) * R + ((c ^ mswz(k + 4)) << 3) + within;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a0));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a1));
        typedef short s16x8 __attribute__((ext_vector_type(8)));
        const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(f16x8, v);
    }
};

template <bool MN, int R, int NT>
struct LoaderSel { using type = KMajorLoader<R, NT>; };
template <int R, int NT>
struct LoaderSel<true, R, NT> { using type = MNMajorLoader<R, NT>; };

__device__ __forceinline__ void decode_tile(int bid, int tiles_n, int sym, int& tm, int& tn) {
    if (!sym) {
        tm = bid / tiles_n;
        tn = bid - tm * tiles_n;
        return;
    }
    // Upper triangle (tm <= tn), row by row.
    int row = 0, left = bid;
    while (left >= tiles_n - row) { left -= tiles_n - row; ++row; }
    tm = row;
    tn = row + left;
}

// Block barrier that orders LDS only.  __syncthreads() is a workgroup fence
// over all address spaces, which on gfx950 also waits for every outstanding
// global load (vmcnt(0)) and so would drain the prefetch of the next K-stage
// at each barrier; the kernel's cross-wave traffic is all in LDS.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Maps the hardware block order (dispatched round-robin over the 8 XCDs) to
// a logical order in which each XCD owns one contiguous range of tiles, so
// neighbouring tiles of a matrix share that XCD's L2.
template <bool STRIPED>
__device__ __forceinline__ void xcd_remap(int& bx, int& by, int& bz) {
    const int gx = gridDim.x, gy = gridDim.y, gz = gridDim.z;
    const int total = gx * gy * gz;
    int lin = bx + gx * (by + gy * bz);
    // Workgroup w runs on XCD w % 8.  The first 8 * floor(total / 8) ids are
    // regrouped so each XCD takes one contiguous run of tiles (sharing
    // operands in its own L2); the ragged tail keeps its order.
    // STRIPED (launches whose matrices differ in cost): each XCD takes whole
    // matrices in turn instead (matrix j of every eight on XCD j % 8), so
    // every XCD gets the same mix of cheap and costly matrices in launch
    // order; the ragged last round keeps its order.
    if constexpr (STRIPED) {
        const int st = gx * gy, full = (gz >> 3) * (st << 3);
        if (lin < full) {
            const int x = lin & 7, j = lin >> 3;
            lin = (j / st) * (st << 3) + x * st + j % st;
        }
    } else {
        const int per = total >> 3;
        if (lin < (per << 3)) lin = (lin & 7) * per + (lin >> 3);
    }
    bx = lin % gx;
    lin /= gx;
    by = lin % gy;
    bz = lin / gy;
}

// At least two waves per SIMD: two 4-wave blocks (or one 8-wave block) per
// CU, so one block's MFMAs overlap the other's LDS and barrier waits.
// MF = 32: v_mfma_f32_32x32x16_f16 blocks (measured issue-bound ceiling on
// gfx950 about 2.4 PFLOP/s, against about 1.45 PFLOP/s for the 16x16x32
// form).
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Epilogues that carry a GramGroups table (grouped Gram launches).
template <class E, class = void>
struct IsGrouped { static constexpr bool value = false; };
template <class E>
struct IsGrouped<E, std::void_t<decltype(std::declval<E>().gg)>> { static constexpr bool value = true; };
// Epilogues that carry a CombineGroups table (grouped Newton-Schulz combines).
template <class E, class = void>
struct IsCmbGrouped { static constexpr bool value = false; };
template <class E>
struct IsCmbGrouped<E, std::void_t<decltype(std::declval<E>().cg)>> { static constexpr bool value = true; };
// Epilogues that carry a SketchGroups table (grouped split-K sketch products).
template <class E, class = void>
struct IsSkGrouped { static constexpr bool value = false; };
template <class E>
struct IsSkGrouped<E, std::void_t<decltype(std::declval<E>().sg)>> { static constexpr bool value = true; };

template <int MF> struct AccSel { using type = f32x4; };
template <> struct AccSel<32> { using type = f32x16; };

template <int BM, int BN, int WM, int WN, int LAYOUT, class Epi, int MF>
__global__ void __launch_bounds__(WM * WN * 64, 2)
gemm_kernel(Operand A, Operand B, GemmShape sh, Epi epi) {
    constexpr int NT = WM * WN * 64;
    constexpr int TM = BM / WM, TN = BN / WN, FM = TM / MF, FN = TN / MF;
    // Accumulators as quads: 4 consecutive rows of one column per lane.
    constexpr int QPB = 4;                          // quads per MFMA block
    static_assert(MF == 32 && TM % MF == 0 && TN % MF == 0, "wave tile must hold whole MFMA blocks");
    constexpr int NQ = FM * FN * QPB;
    // Two LDS stages: the MFMAs of stage i overlap the LDS stores of stage
    // i + 1 and the global loads of stage i + 2.  The epilogue reuses the
    // same LDS to stage one wave-row of fp32 results (row stride BN + 4).
    constexpr int kStageBytes = 2 * (BM + BN) * BK * 2;
    // Result rows staged per epilogue pass: the whole tile when its fp32
    // staging adds little to the operand stages (up to 128 x 128), else 64
    // rows, so that the fp32 staging and the fp16 transpose of the mirror
    // (BN x 64 halves, after it in LDS) fit next to each other.
    constexpr int kEpiRows = BM * BN <= 128 * 128 ? BM : 64;
    constexpr int kEpiBytes = kEpiRows * (BN + 4) * 4;
    // Symmetric results write their mirror from an LDS transpose of the fp16
    // tile: src is symmetric wherever the result is (A for B = b A + c A^2,
    // the right factor of a Gram-space product), so the mirrored values are
    // exactly the transposed results.
    constexpr bool kSepMirror = Epi::kind == EpiKind::Affine && BM * BN > 128 * 128;  // buffer after the staging
    constexpr int kMirrorOff = (kEpiBytes + 15) / 16 * 16;
    static_assert(!kSepMirror || kMirrorOff + BN * kEpiRows * 2 <= kStageBytes, "mirror buffer does not fit");
    __shared__ __attribute__((aligned(16))) unsigned char smem[kStageBytes > kEpiBytes ? kStageBytes : kEpiBytes];
    __shared__ float red[NT / 64];
    half_t* const sbase = reinterpret_cast<half_t*>(smem);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave - (wave / WN) * WN;
    int bx = blockIdx.x, split = blockIdx.y, z = blockIdx.z;
    xcd_remap<IsGrouped<Epi>::value || IsSkGrouped<Epi>::value || IsCmbGrouped<Epi>::value>(bx, split, z);
    if constexpr (Epi::kind == EpiKind::ApplyNorm) {
        if (epi.need && epi.need[z] == 0) return;   // whole block, before any barrier
    }
    int tiles_n = sh.N / BN, K = sh.K, k_chunk = sh.k_chunk;
    int sgi = 0, slz = 0;           // sketch group and matrix within it
    if constexpr (IsSkGrouped<Epi>::value) {
        while (sgi + 1 < epi.sg.n && z >= epi.sg.zbeg[sgi + 1]) ++sgi;
        slz = z - epi.sg.zbeg[sgi];
        tiles_n = epi.sg.N[sgi] / BN;
        // The grid spans the largest group; the whole block leaves before
        // its first barrier when its tile or split is past this group's.
        if (bx >= (sh.M / BM) * tiles_n || split >= epi.sg.splits[sgi]) return;
        K = epi.sg.K[sgi];
        k_chunk = epi.sg.k_chunk[sgi];
    }
    int cgi = 0, clz = 0;           // combine group and matrix within it
    if constexpr (IsCmbGrouped<Epi>::value) {
        while (cgi + 1 < epi.cg.n && z >= epi.cg.zbeg[cgi + 1]) ++cgi;
        clz = z - epi.cg.zbeg[cgi];
        tiles_n = epi.cg.N[cgi] / BN;
        if (bx >= (sh.M / BM) * tiles_n) return;   // whole block, before any barrier
    }
    int tm, tn;
    decode_tile(bx, tiles_n, sh.sym, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = split * k_chunk;
    int kend = min(K, kbeg + k_chunk);

    const half_t* Ab = A.ptr + (int64_t)z * A.batch_stride;
    const half_t* Bb = B.ptr + (int64_t)z * B.batch_stride;
    int64_t lda = A.ld, ldb = B.ld;
    int zo = z;                      // output matrix index
    const float* mulz = nullptr;     // this matrix's scale pair, or null
    if constexpr (IsGrouped<Epi>::value) {
        int g = 0;
        while (g + 1 < epi.gg.n && z >= epi.gg.zbeg[g + 1]) ++g;
        const int lz = z - epi.gg.zbeg[g];
        Ab = epi.gg.x[g] + (int64_t)lz * epi.gg.stride[g];
        Bb = Ab;
        lda = ldb = epi.gg.ld[g];
        kend = epi.gg.K[g];
        zo = epi.gg.zout[g] + lz;
        mulz = epi.gg.mul[g] ? epi.gg.mul[g] + 2 * lz : nullptr;
    } else if constexpr (IsCmbGrouped<Epi>::value) {
        Ab = epi.cg.a[cgi] + (int64_t)clz * epi.cg.a_stride[cgi];
        Bb = epi.cg.b[cgi] + (int64_t)clz * epi.cg.b_stride[cgi];
        lda = epi.cg.lda[cgi];
        ldb = epi.cg.ldb[cgi];
        zo = clz;
        mulz = epi.cg.mul[cgi] ? epi.cg.mul[cgi] + 2 * clz : nullptr;
    } else if constexpr (IsSkGrouped<Epi>::value) {
        Ab = epi.sg.a[sgi] + (int64_t)slz * epi.sg.a_stride[sgi];
        Bb = epi.sg.b[sgi] + (int64_t)slz * epi.sg.b_stride[sgi];
        lda = epi.sg.lda[sgi];
        ldb = epi.sg.ldb[sgi];
    } else if constexpr (Epi::kind == EpiKind::Affine) {
        mulz = epi.mul ? epi.mul + 2 * z : nullptr;
    }
    // Per-matrix operands of the Affine and ApplyNorm epilogues (the grouped
    // combine takes them from its table).
    half_t* e_out = nullptr;
    const half_t* e_src = nullptr;
    int64_t e_ld_out = 0, e_stride_out = 0, e_ld_src = 0, e_stride_src = 0;
    float* e_sumsq = nullptr;
    int e_tiles = 0;
    if constexpr (IsCmbGrouped<Epi>::value) {
        e_out = epi.cg.out[cgi];
        e_ld_out = epi.cg.ld_out[cgi];
        e_stride_out = epi.cg.stride_out[cgi];
        e_src = epi.cg.src[cgi];
        e_ld_src = epi.cg.ld_src[cgi];
        e_stride_src = epi.cg.stride_src[cgi];
        e_sumsq = epi.cg.sumsq[cgi];
        e_tiles = epi.cg.tiles[cgi];
    } else if constexpr (Epi::kind == EpiKind::Affine) {
        e_out = epi.out;
        e_ld_out = epi.ld_out;
        e_stride_out = epi.stride_out;
        e_src = epi.src;
        e_ld_src = epi.ld_src;
        e_stride_src = epi.stride_src;
        e_sumsq = epi.sumsq;
        e_tiles = epi.tiles_per_mat;
    } else if constexpr (Epi::kind == EpiKind::ApplyNorm) {
        e_sumsq = epi.sumsq;
        e_tiles = epi.tiles_per_mat;
    }
    using LA = typename LoaderSel<(LAYOUT == 2), BM, NT>::type;
    using LB = typename LoaderSel<(LAYOUT >= 1), BN, NT>::type;
    // DEEP: two staging sets, so each K-step's global loads have two
    // K-steps to arrive (covers L2 misses served from the Infinity Cache);
    // the tiles up to 128 x 128 have the registers for it, and so has the
    // 64 x 512 one (eight waves: the same loads per thread as 64 x 256).
    constexpr bool DEEP = MF == 32 && (BM * BN <= 128 * 128 || (BM == 64 && BN == 512));
    u32x4 ra[LA::N], rb[LB::N];
    u32x4 ra2[LA::N], rb2[LB::N];

    using AccT = typename AccSel<MF>::type;
    AccT acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = AccT{};

    // One K-step with 32x32x16 MFMAs (BK / 16 sub-steps).  With STORE the next
    // stage's staging registers go to LDS and, with LOAD, the stage after
    // that is fetched into them; staging item i is stored (and refilled) at
    // sub-step i * NSUB / N, and the scheduling groups below interleave one
    // MFMA with one LDS or global access so the memory traffic of the step
    // is issued between its MFMAs.
    constexpr int NSUB = BK / 16;
    auto kstep32 = [&](auto store_tag, auto load_tag, int stage, int k_load, auto& rA, auto& rB) {
        constexpr bool STORE = decltype(store_tag)::value, LOAD = decltype(load_tag)::value;
        const half_t* ca = sbase + stage * (BM + BN) * BK;
        const half_t* cb = ca + BM * BK;
        half_t* sa = sbase + (stage ^ 1) * (BM + BN) * BK;
        half_t* sb = sa + BM * BK;
        f16x8 af[2][FM], bf[2][FN];
        auto read_frags = [&](int s, int buf) {
#pragma unroll
            for (int i = 0; i < FM; ++i) af[buf][i] = LA::frag(ca, wm * TM + i * 32, s, lane);
#pragma unroll
            for (int j = 0; j < FN; ++j) bf[buf][j] = LB::frag(cb, wn * TN + j * 32, s, lane);
        };
        read_frags(0, 0);
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
            if (s + 1 < NSUB) read_frags(s + 1, (s + 1) & 1);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[s & 1][i], bf[s & 1][j], acc[i][j], 0, 0, 0);
            if constexpr (STORE) {
#pragma unroll
                for (int it = 0; it < LA::N; ++it)
                    if (it * NSUB / LA::N == s) {
                        LA::store_item(rA, sa, tid, it);
                        if constexpr (LOAD) LA::load_item(rA, Ab, lda, m0, k_load, tid, it);
                    }
#pragma unroll
                for (int it = 0; it < LB::N; ++it)
                    if (it * NSUB / LB::N == s) {
                        LB::store_item(rB, sb, tid, it);
                        if constexpr (LOAD) LB::load_item(rB, Bb, ldb, n0, k_load, tid, it);
                    }
            }
        }
        // Issue order: the fragments of sub-step 0, then per sub-step each
        // MFMA followed by one fragment read of the next sub-step or, once
        // those are out, one LDS store (and its refill load).  An MN-major
        // fragment is two reads.
        constexpr int RD = (LA::kTrans ? 2 : 1) * FM + (LB::kTrans ? 2 : 1) * FN;
        __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
            int nw = 0;
#pragma unroll
            for (int it = 0; it < LA::N; ++it) nw += (it * NSUB / LA::N == s);
#pragma unroll
            for (int it = 0; it < LB::N; ++it) nw += (it * NSUB / LB::N == s);
            if (!STORE) nw = 0;
            const int nr = s + 1 < NSUB ? RD : 0;
            const int per = (nr + FM * FN - 1) / (FM * FN);     // 0, 1 or 2
            int r_left = nr, w_left = nw;
#pragma unroll
            for (int i = 0; i < FM * FN; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (r_left >= 2 && per == 2) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                    r_left -= 2;
                } else if (r_left > 0) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    --r_left;
                } else if (w_left > 0) {
                    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
                    if (LOAD) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                    --w_left;
                }
            }
#pragma unroll
            for (int q = 0; q < LA::N + LB::N; ++q)
                if (q < w_left) {
                    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
                    if (LOAD) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                }
        }
    };
    using T_ = std::true_type;
    using F_ = std::false_type;

    if (kbeg < kend && DEEP) {
        // Step j computes LDS stage j & 1, stores staging set j & 1 (data of
        // step j + 1) into the other stage and refills that set with the
        // data of step j + 3 (clamped to the last K-step near the end: such
        // loads are never stored).  Unrolled by two so the set is static.
        const int nk = (kend - kbeg) / BK;
        auto kat = [&](int j) { return kbeg + min(j, nk - 1) * BK; };
        LA::load(ra, Ab, lda, m0, kbeg, tid);
        LB::load(rb, Bb, ldb, n0, kbeg, tid);
        LA::store(ra, sbase, tid);
        LB::store(rb, sbase + BM * BK, tid);
        LA::load(ra, Ab, lda, m0, kat(1), tid);
        LB::load(rb, Bb, ldb, n0, kat(1), tid);
        LA::load(ra2, Ab, lda, m0, kat(2), tid);
        LB::load(rb2, Bb, ldb, n0, kat(2), tid);
        int j = 0;
        for (; j + 2 < nk; j += 2) {
            lds_barrier();
            kstep32(T_{}, T_{}, 0, kat(j + 3), ra, rb);
            lds_barrier();
            kstep32(T_{}, T_{}, 1, kat(j + 4), ra2, rb2);
        }
        if (j + 1 < nk) {
            lds_barrier();
            kstep32(T_{}, F_{}, 0, 0, ra, rb);
            ++j;
        }
        lds_barrier();
        kstep32(F_{}, F_{}, j & 1, 0, ra, rb);
    } else if (kbeg < kend) {
        LA::load(ra, Ab, lda, m0, kbeg, tid);
        LB::load(rb, Bb, ldb, n0, kbeg, tid);
        LA::store(ra, sbase, tid);
        LB::store(rb, sbase + BM * BK, tid);
        if (kbeg + BK < kend) {
            LA::load(ra, Ab, lda, m0, kbeg + BK, tid);
            LB::load(rb, Bb, ldb, n0, kbeg + BK, tid);
        }
        // Branch-free steady state, the last two K-steps peeled.
        int stage = 0;
        int k0 = kbeg;
        for (; k0 + 2 * BK < kend; k0 += BK, stage ^= 1) {
            lds_barrier();
            kstep32(T_{}, T_{}, stage, k0 + 2 * BK, ra, rb);
        }
        if (k0 + BK < kend) {
            lds_barrier();
            kstep32(T_{}, F_{}, stage, 0, ra, rb);
            k0 += BK;
            stage ^= 1;
        }
        lds_barrier();
        kstep32(F_{}, F_{}, stage, 0, ra, rb);
    }

    // Quad qi of this lane: rows quad_row(qi) + 0..3 (relative to the wave
    // tile), column quad_col(qi): register r of 32x32 block (i, j) is
    // row 32i + 8*(r/4) + 4*(lane/32) + r%4, column 32j + lane%32.
    auto quad_row = [&](int qi) -> int {
        const int blk = qi / QPB, g = qi - blk * QPB, i = blk / FN;
        return 32 * i + 8 * g + 4 * (lane >> 5);
    };
    auto quad_col = [&](int qi) -> int {
        const int blk = qi / QPB, j = blk - (blk / FN) * FN;
        return 32 * j + (lane & 31);
    };
    auto quad_val = [&](int qi, int r) -> float {
        const int blk = qi / QPB, g = qi - blk * QPB, i = blk / FN, j = blk - i * FN;
        return acc[i][j][4 * g + r];
    };
    const int rw0 = m0 + wm * TM, cw0 = n0 + wn * TN;

    if constexpr (Epi::kind == EpiKind::Partial) {
        float* out;
        int64_t ldo;
        if constexpr (IsSkGrouped<Epi>::value) {
            ldo = epi.sg.N[sgi];
            float* const o32 = epi.sg.out32[sgi];
            half_t* const o16 = epi.sg.out16[sgi];
            if (epi.sg.splits[sgi] == 1 && (o32 || o16)) {
                // One split: the final product, as the split reduction
                // would write it.
                const int64_t zoff = (int64_t)slz * epi.sg.stride_out[sgi];
                const float sc16 = epi.sg.scale16[sgi];
#pragma unroll
                for (int qi = 0; qi < NQ; ++qi)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int64_t idx = zoff + (int64_t)(rw0 + quad_row(qi) + r) * ldo + cw0 + quad_col(qi);
                        const float v = quad_val(qi, r);
                        if (o32) o32[idx] = v;
                        if (o16) o16[idx] = (half_t)(v * sc16);
                    }
                return;
            }
            out = epi.sg.out[sgi] + (int64_t)slz * epi.sg.stride_mat[sgi] + (int64_t)split * epi.sg.stride_split[sgi];
        } else {
            out = epi.out + (int64_t)z * epi.stride_mat + (int64_t)split * epi.stride_split;
            ldo = epi.ld_out;
        }
#pragma unroll
        for (int qi = 0; qi < NQ; ++qi)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[(int64_t)(rw0 + quad_row(qi) + r) * ldo + cw0 + quad_col(qi)] = quad_val(qi, r);
        return;
    } else {
        // Per-epilogue set-up.
        float ca = 1.f, cs = 0.f, scale = 0.f;
        half_t* out = nullptr;
        const half_t* src = nullptr;
        const half_t* psi = nullptr;
        float* w = nullptr;
        bool mirror = false;
        if constexpr (Epi::kind == EpiKind::Affine) {
            float mul = 1.f;
            if (mulz && epi.mul_pow > 0) {
                const float f = mulz[0];
                mul = epi.mul_pow == 1 ? f : f * f;
            }
            ca = epi.ca * mul;
            cs = epi.cs * mul;
            out = e_out + (int64_t)zo * e_stride_out;
            src = e_src ? e_src + (int64_t)zo * e_stride_src : nullptr;
            // Off-diagonal tiles of a symmetric result also write their
            // transpose (through LDS, after each pass's row stores).
            mirror = sh.sym && tm != tn;
        } else {
            psi = epi.psi + (int64_t)z * epi.stride_psi;
            if constexpr (Epi::kind == EpiKind::Apply) {
                const float t2 = epi.tnorm2[z];
                scale = t2 > 0.f ? epi.target_rms * sqrtf((float)epi.rows * (float)epi.cols) / sqrtf(t2) : 0.f;
                w = epi.ptrs.w[z];
            }
        }
        // Stage PR rows of fp32 results at a time in LDS (the whole tile at
        // once when it fits, else one wave-row per pass), then walk them
        // row-contiguously: 8 columns per item (16-byte fp16 accesses).
        constexpr int LDST = BN + 4;
        constexpr int C8 = BN / 8;
        constexpr int PR = kEpiRows;
        float* stg = reinterpret_cast<float*>(smem);
        float ss = 0.f;
#pragma unroll 1
        for (int pass = 0; pass < BM / PR; ++pass) {
            constexpr int ITEMS = (PR * C8 + NT - 1) / NT;
            // Affine: this pass's src rows are loaded before the staging
            // barriers, so their latency overlaps the LDS traffic.
            constexpr int SB = Epi::kind == EpiKind::Affine && !IsGrouped<Epi>::value ? ITEMS : 1;
            u32x4 sbuf[SB];
            if constexpr (Epi::kind == EpiKind::Affine) {
                if (src) {
#pragma unroll
                    for (int q = 0; q < SB; ++q) {
                        const int c = tid + q * NT;
                        if (c < PR * C8) {
                            const int r = c / C8, c8 = (c - r * C8) * 8;
                            sbuf[q] = *reinterpret_cast<const u32x4*>(src + (int64_t)(m0 + pass * PR + r) * e_ld_src +
                                                                      n0 + c8);
                        }
                    }
                }
            }
            lds_barrier();
            // This pass's rows [pass * PR, pass * PR + PR) of the tile (a
            // quad's four rows never straddle a pass).
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi) {
                const int qrow = wm * TM + quad_row(qi) - pass * PR;
                if (qrow >= 0 && qrow < PR) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) stg[(qrow + r) * LDST + wn * TN + quad_col(qi)] = quad_val(qi, r);
                }
            }
            lds_barrier();
            if constexpr (Epi::kind == EpiKind::Apply || Epi::kind == EpiKind::ApplyNorm) {
                // Issue every item's Psi (and W) loads before using any of them.
                u32x4 pbuf[ITEMS];
                f32x4 wbuf[ITEMS][2];
                bool okv[ITEMS];
#pragma unroll
                for (int it = 0; it < ITEMS; ++it) {
                    const int c = tid + it * NT;
                    const int r = c / C8, c8 = (c - r * C8) * 8;
                    const int grow = m0 + pass * PR + r, gcol = n0 + c8;
                    okv[it] = c < PR * C8 && grow < epi.rows && gcol < epi.cols;
                    if (okv[it]) {
                        pbuf[it] = *reinterpret_cast<const u32x4*>(psi + (int64_t)grow * epi.ld_psi + gcol);
                        if constexpr (Epi::kind == EpiKind::Apply) {
                            if (gcol + 8 <= epi.cols && epi.vec_ok) {
                                const float* wp = w + (int64_t)grow * epi.cols + gcol;
                                wbuf[it][0] = *reinterpret_cast<const f32x4*>(wp);
                                wbuf[it][1] = *reinterpret_cast<const f32x4*>(wp + 4);
                            }
                        }
                    }
                }
#pragma unroll
                for (int it = 0; it < ITEMS; ++it) {
                    if (!okv[it]) continue;
                    const int c = tid + it * NT;
                    const int r = c / C8, c8 = (c - r * C8) * 8;
                    const int grow = m0 + pass * PR + r, gcol = n0 + c8;
                    const f32x4 lo = *reinterpret_cast<const f32x4*>(stg + r * LDST + c8);
                    const f32x4 hi = *reinterpret_cast<const f32x4*>(stg + r * LDST + c8 + 4);
                    const half_t* pv = reinterpret_cast<const half_t*>(&pbuf[it]);
                    float t[8];
#pragma unroll
                    for (int e = 0; e < 4; ++e) { t[e] = (float)pv[e] + lo[e]; t[e + 4] = (float)pv[e + 4] + hi[e]; }
                    const bool full = gcol + 8 <= epi.cols;
                    if constexpr (Epi::kind == EpiKind::ApplyNorm) {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (full || gcol + e < epi.cols) ss = fmaf(t[e], t[e], ss);
                    } else {
                        float* wp = w + (int64_t)grow * epi.cols + gcol;
                        if (full && epi.vec_ok) {
                            f32x4 w0 = wbuf[it][0], w1 = wbuf[it][1];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                w0[e] = w0[e] - epi.lr * (scale * t[e] + epi.wd * w0[e]);
                                w1[e] = w1[e] - epi.lr * (scale * t[e + 4] + epi.wd * w1[e]);
                            }
                            *reinterpret_cast<f32x4*>(wp) = w0;
                            *reinterpret_cast<f32x4*>(wp + 4) = w1;
                        } else {
#pragma unroll
                            for (int e = 0; e < 8; ++e)
                                if (gcol + e < epi.cols) {
                                    const float wv = wp[e];
                                    wp[e] = wv - epi.lr * (scale * t[e] + epi.wd * wv);
                                }
                        }
                    }
                }
                continue;
            }
            u32x4 hk[kSepMirror ? 1 : ITEMS];      // fp16 results, kept for the mirror
            half_t* const tb = reinterpret_cast<half_t*>(smem + (kSepMirror ? kMirrorOff : 0));
            constexpr int R8 = PR / 8;
#pragma unroll
            for (int it = 0; it < ITEMS; ++it) {
                const int c = tid + it * NT;
                if (c >= PR * C8) break;
                const int r = c / C8, c8 = (c - r * C8) * 8;
                const int grow = m0 + pass * PR + r, gcol = n0 + c8;
                const f32x4 lo = *reinterpret_cast<const f32x4*>(stg + r * LDST + c8);
                const f32x4 hi = *reinterpret_cast<const f32x4*>(stg + r * LDST + c8 + 4);
                float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                if constexpr (Epi::kind == EpiKind::Affine) {
                    const half_t* sv = reinterpret_cast<const half_t*>(&sbuf[it < SB ? it : 0]);
                    half_t hv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        float x = ca * v[e];
                        if (src) x += cs * (float)sv[e];
                        hv[e] = (half_t)x;
                        const float q = (float)hv[e];
                        ss += q * q;
                    }
                    // Streamed past L2 (nontemporal): the result is read by a
                    // later launch, and keeping it out of L2 leaves the
                    // operand panels resident.
                    const u32x4 hq = *reinterpret_cast<const u32x4*>(hv);
                    if constexpr (kSepMirror) {
                        // Transposed copy straight into its own LDS buffer.
                        if (mirror) {
#pragma unroll
                            for (int e = 0; e < 8; ++e) {
                                const int cc = c8 + e;
                                tb[cc * PR + (((r >> 3) ^ ((cc >> 3) & (R8 - 1))) << 3) + (r & 7)] = hv[e];
                            }
                        }
                    } else {
                        hk[it] = hq;
                    }
                    __builtin_nontemporal_store(hq, reinterpret_cast<u32x4*>(out + (int64_t)grow * e_ld_out + gcol));
                }
            }
            if constexpr (Epi::kind == EpiKind::Affine) {
                if (mirror) {
                    // T[c][r] = result[r][c] for this pass's PR rows: row c of
                    // T holds PR halves in chunks of 8, chunk j stored at
                    // j ^ (c / 8 mod PR / 8) so the 2-byte writes of one
                    // wave spread over the banks; then 16-byte rows out.  The
                    // whole-tile pass (128 x 128) transposes its fp16 results
                    // from registers into the freed staging LDS; the 64-row
                    // passes of the larger tile wrote theirs above.
                    lds_barrier();
#pragma unroll
                    for (int it = 0; it < (kSepMirror ? 0 : ITEMS); ++it) {
                        const int c = tid + it * NT;
                        if (c >= PR * C8) break;
                        const int r = c / C8, c8 = (c - r * C8) * 8;
                        const half_t* hv = reinterpret_cast<const half_t*>(&hk[it]);
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int cc = c8 + e;
                            tb[cc * PR + (((r >> 3) ^ ((cc >> 3) & (R8 - 1))) << 3) + (r & 7)] = hv[e];
                        }
                    }
                    lds_barrier();
                    for (int q = tid; q < BN * R8; q += NT) {
                        const int cc = q / R8, j = q - cc * R8;
                        const u32x4 v = *reinterpret_cast<const u32x4*>(tb + cc * PR + ((j ^ ((cc >> 3) & (R8 - 1))) << 3));
                        __builtin_nontemporal_store(
                            v, reinterpret_cast<u32x4*>(out + (int64_t)(n0 + cc) * e_ld_out + m0 + pass * PR + 8 * j));
                    }
                }
            }
        }
        const bool want_sum = (Epi::kind == EpiKind::ApplyNorm) ||
                              (Epi::kind == EpiKind::Affine && e_sumsq != nullptr);
        if (want_sum) {
            ss = wave_sum(ss);
            lds_barrier();
            if (lane == 0) red[wave] = ss;
            lds_barrier();
            if (tid == 0) {
                float t = 0.f;
                for (int q = 0; q < NT / 64; ++q) t += red[q];
                e_sumsq[(int64_t)zo * e_tiles + bx] = t;
            }
        }
    }
}

struct EAff : EpiAffine { static constexpr EpiKind kind = EpiKind::Affine; };
struct EAffG : EpiAffine {
    static constexpr EpiKind kind = EpiKind::Affine;
    GramGroups gg;
};
struct EPar : EpiPartial { static constexpr EpiKind kind = EpiKind::Partial; };
struct EAffC : EpiAffine {
    static constexpr EpiKind kind = EpiKind::Affine;
    CombineGroups cg;
};
struct EParG : EpiPartial {
    static constexpr EpiKind kind = EpiKind::Partial;
    SketchGroups sg;
};
struct EApp : EpiApplyUpdate { static constexpr EpiKind kind = EpiKind::Apply; };
struct EAppN : EpiApplyNorm { static constexpr EpiKind kind = EpiKind::ApplyNorm; };

thread_local hipEvent_t t_ev_start = nullptr, t_ev_stop = nullptr;

bool take_launch_events(hipEvent_t& start, hipEvent_t& stop) {
    if (!t_ev_start) return false;
    start = t_ev_start;
    stop = t_ev_stop;
    t_ev_start = t_ev_stop = nullptr;
    return true;
}

template <int BM, int BN, int WM, int WN, int LAYOUT, class E, int MF = 32>
hipError_t run(Operand A, Operand B, GemmShape sh, int batch, const E& e, hipStream_t s) {
    if (sh.M % BM || sh.N % BN || sh.K % BK || sh.k_chunk % BK || batch < 1) return hipErrorInvalidValue;
    const int tm = sh.M / BM, tn = sh.N / BN;
    int tiles = tm * tn;
    if (sh.sym) {
        if (tm != tn) return hipErrorInvalidValue;
        tiles = tn * (tn + 1) / 2;
    }
    dim3 grid(tiles, sh.k_split, batch);
    hipEvent_t ev0, ev1;
    if (take_launch_events(ev0, ev1))
        hipExtLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, LAYOUT, E, MF>), grid, dim3(WM * WN * 64), 0, s, ev0, ev1, 0,
                              A, B, sh, e);
    else
        hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, LAYOUT, E, MF>), grid, dim3(WM * WN * 64), 0, s, A, B, sh, e);
    return hipGetLastError();
}

template <class E, int LAYOUT>
hipError_t dispatch_cfg(TileCfg cfg, Operand A, Operand B, GemmShape sh, int batch, const E& e, hipStream_t s) {
    switch (cfg) {
        case TileCfg::Big:       return run<128, 128, 2, 2, LAYOUT>(A, B, sh, batch, e, s);
        case TileCfg::Skinny64:  return run<64, 256, 1, 4, LAYOUT>(A, B, sh, batch, e, s);
        case TileCfg::Skinny64W: return run<64, 512, 1, 8, LAYOUT>(A, B, sh, batch, e, s);
        case TileCfg::Skinny128: return run<128, 256, 2, 4, LAYOUT>(A, B, sh, batch, e, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

void arm_launch_events(hipEvent_t start, hipEvent_t stop) {
    t_ev_start = start;
    t_ev_stop = stop;
}
bool disarm_launch_events() {
    const bool armed = t_ev_start != nullptr;
    t_ev_start = t_ev_stop = nullptr;
    return armed;
}

int gemm_tile_m(TileCfg cfg) {
    switch (cfg) {
        case TileCfg::Big: return 128;
        case TileCfg::Big256: return 256;
        case TileCfg::Skinny64: return 64;
        case TileCfg::Skinny64W: return 64;
        case TileCfg::Skinny128: return 128;
        case TileCfg::Apply: return 64;
    }
    return 0;
}
int gemm_tile_n(TileCfg cfg) {
    switch (cfg) {
        case TileCfg::Skinny64W: return 512;
        case TileCfg::Big: return 128;
        case TileCfg::Apply: return 128;
        default: return 256;
    }
}

hipError_t launch_gemm_affine(TileCfg cfg, int layout, Operand A, Operand B, GemmShape sh,
                              int batch, const EpiAffine& e, hipStream_t s) {
    EAff ee;
    static_cast<EpiAffine&>(ee) = e;
    if (cfg == TileCfg::Big) {
        switch (layout) {
            case 0: return run<128, 128, 2, 2, 0>(A, B, sh, batch, ee, s);
            case 1: return run<128, 128, 2, 2, 1>(A, B, sh, batch, ee, s);
            case 2: return run<128, 128, 2, 2, 2>(A, B, sh, batch, ee, s);
        }
    } else if (cfg == TileCfg::Big256) {
        // (Layout 2 on this tile serves the grouped Gram only.)
        switch (layout) {
            case 0: return run<256, 256, 2, 4, 0, EAff, 32>(A, B, sh, batch, ee, s);
            case 1: return run<256, 256, 2, 4, 1, EAff, 32>(A, B, sh, batch, ee, s);
        }
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_gram_grouped(TileCfg cfg, int layout, const GramGroups& g, int sp, const EpiAffine& e,
                                    hipStream_t s) {
    if (g.n < 1 || g.n > kMaxGramGroups || (layout != 0 && layout != 2)) return hipErrorInvalidValue;
    int kmax = 0;
    for (int i = 0; i < g.n; ++i) {
        if (g.K[i] < BK || g.K[i] % BK || g.zbeg[i + 1] <= g.zbeg[i]) return hipErrorInvalidValue;
        kmax = std::max(kmax, g.K[i]);
    }
    EAffG ee;
    static_cast<EpiAffine&>(ee) = e;
    ee.mul = nullptr;
    ee.gg = g;
    Operand dummy{g.x[0], g.ld[0], 0};
    GemmShape sh{sp, sp, kmax, 1, kmax, 1};
    const int batch = g.zbeg[g.n] - g.zbeg[0];
    if (g.zbeg[0] != 0) return hipErrorInvalidValue;
    if (layout == 0) {
        if (cfg == TileCfg::Big) return run<128, 128, 2, 2, 0, EAffG>(dummy, dummy, sh, batch, ee, s);
        if (cfg == TileCfg::Big256) return run<256, 256, 2, 4, 0, EAffG>(dummy, dummy, sh, batch, ee, s);
    } else {
        if (cfg == TileCfg::Big) return run<128, 128, 2, 2, 2, EAffG>(dummy, dummy, sh, batch, ee, s);
        if (cfg == TileCfg::Big256) return run<256, 256, 2, 4, 2, EAffG>(dummy, dummy, sh, batch, ee, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_partial(TileCfg cfg, int layout, Operand A, Operand B, GemmShape sh,
                               int batch, const EpiPartial& e, hipStream_t s) {
    EPar ee;
    static_cast<EpiPartial&>(ee) = e;
    if (cfg != TileCfg::Skinny64 && cfg != TileCfg::Skinny64W && cfg != TileCfg::Skinny128)
        return hipErrorInvalidValue;
    switch (layout) {
        case 0: return dispatch_cfg<EPar, 0>(cfg, A, B, sh, batch, ee, s);
        case 1: return dispatch_cfg<EPar, 1>(cfg, A, B, sh, batch, ee, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_partial_grouped(TileCfg cfg, int layout, int M, const SketchGroups& g, hipStream_t s) {
    if (cfg != TileCfg::Skinny64 && cfg != TileCfg::Skinny64W && cfg != TileCfg::Skinny128)
        return hipErrorInvalidValue;
    if (g.n < 1 || g.n > kMaxItems || g.zbeg[0] != 0 || (layout != 0 && layout != 1)) return hipErrorInvalidValue;
    const int bm = gemm_tile_m(cfg), bn = gemm_tile_n(cfg);
    if (M < bm || M % bm) return hipErrorInvalidValue;
    int maxN = 0, maxS = 0;
    for (int i = 0; i < g.n; ++i) {
        if (g.zbeg[i + 1] <= g.zbeg[i] || g.N[i] < bn || g.N[i] % bn || g.K[i] < BK || g.K[i] % BK ||
            g.k_chunk[i] < BK || g.k_chunk[i] % BK || g.splits[i] < 1 ||
            (int64_t)(g.splits[i] - 1) * g.k_chunk[i] >= g.K[i] || (int64_t)g.splits[i] * g.k_chunk[i] < g.K[i])
            return hipErrorInvalidValue;
        maxN = std::max(maxN, g.N[i]);
        maxS = std::max(maxS, g.splits[i]);
    }
    EParG ee{};
    ee.sg = g;
    // The grid spans the largest group (its tiles, its splits); operands
    // and strides come from the table.
    Operand dummy{nullptr, 0, 0};
    GemmShape sh{M, maxN, BK, maxS, BK, 0};
    switch (layout) {
        case 0: return dispatch_cfg<EParG, 0>(cfg, dummy, dummy, sh, g.zbeg[g.n], ee, s);
        case 1: return dispatch_cfg<EParG, 1>(cfg, dummy, dummy, sh, g.zbeg[g.n], ee, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_combine_grouped(TileCfg cfg, int s_dim, const CombineGroups& g, const EpiAffine& e,
                                       hipStream_t s) {
    if (cfg != TileCfg::Big && cfg != TileCfg::Big256) return hipErrorInvalidValue;
    if (g.n < 1 || g.n > kMaxItems || g.zbeg[0] != 0) return hipErrorInvalidValue;
    const int t = cfg == TileCfg::Big256 ? 256 : 128;
    if (s_dim < t || s_dim % t) return hipErrorInvalidValue;
    int maxN = 0;
    for (int i = 0; i < g.n; ++i) {
        if (g.zbeg[i + 1] <= g.zbeg[i] || g.N[i] < t || g.N[i] % t) return hipErrorInvalidValue;
        if (g.sumsq[i] && g.tiles[i] != (s_dim / t) * (g.N[i] / t)) return hipErrorInvalidValue;
        maxN = std::max(maxN, g.N[i]);
    }
    EAffC ee{};
    static_cast<EpiAffine&>(ee) = e;
    ee.cg = g;
    // The grid spans the widest group; operands, outputs and scales come
    // from the table.
    Operand dummy{nullptr, 0, 0};
    GemmShape sh{s_dim, maxN, s_dim, 1, s_dim, 0};
    if (cfg == TileCfg::Big) return run<128, 128, 2, 2, 1>(dummy, dummy, sh, g.zbeg[g.n], ee, s);
    return run<256, 256, 2, 4, 1, EAffC, 32>(dummy, dummy, sh, g.zbeg[g.n], ee, s);
}

hipError_t launch_gemm_gram_f32(int layout, Operand A, Operand B, GemmShape sh, int batch, const EpiPartial& e,
                                hipStream_t s) {
    EPar ee;
    static_cast<EpiPartial&>(ee) = e;
    if (layout == 0) return run<128, 128, 2, 2, 0>(A, B, sh, batch, ee, s);
    if (layout == 2) return run<128, 128, 2, 2, 2>(A, B, sh, batch, ee, s);
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_apply(Operand A, Operand B, GemmShape sh, int batch,
                             const EpiApplyUpdate& e, hipStream_t s) {
    EApp ee;
    static_cast<EpiApplyUpdate&>(ee) = e;
    return run<64, 128, 1, 4, 0>(A, B, sh, batch, ee, s);
}

hipError_t launch_gemm_apply_norm(Operand A, Operand B, GemmShape sh, int batch,
                                  const EpiApplyNorm& e, hipStream_t s) {
    EAppN ee;
    static_cast<EpiApplyNorm&>(ee) = e;
    return run<64, 128, 1, 4, 0>(A, B, sh, batch, ee, s);
}

}  // namespace np
