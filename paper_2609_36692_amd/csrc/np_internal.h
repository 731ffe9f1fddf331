// Internal declarations shared by the host driver and the gfx950 kernels of
// the NormPre library.  Not part of the public ABI (that is include/normpre.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace np {

typedef _Float16 half_t;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Every workspace matrix is padded with zeros to a multiple of this many
// rows and columns, so the MFMA kernels never see a ragged tile.  Zero
// padding is exact for every product in the step: padded rows/columns of
// Psi are zero, and the Newton-Schulz map sends a zero block to zero.
constexpr int kPad = 256;
// The sketch width l is padded to a multiple of this (MFMA K granule).
constexpr int kEllPad = 64;
// Grouped launches over the items of one pool (same l): item g covers the
// launch's matrices [zbeg[g], zbeg[g + 1]), which are also its matrices'
// indices in the pool's l x l buffers.
constexpr int kMaxItems = 8;

inline int64_t round_up(int64_t x, int64_t g) { return (x + g - 1) / g * g; }

// Matrices handled by one launch that touches caller memory (W, G, M):
// pointers travel in the kernel arguments, so no host-to-device copy is
// ever needed inside a step.
constexpr int kChunk = 32;
struct PtrChunk {
    float* w[kChunk];
    float* m[kChunk];
    const float* g[kChunk];
};

// ---------------------------------------------------------------- GEMM ---
// C(mm, nn) = sum_k Aop(mm, k) * Bop(nn, k) in fp16 x fp16 -> fp32 MFMA.
// K-major operand:  op(r, k) = ptr[r * ld + k]
// MN-major operand: op(r, k) = ptr[k * ld + r]
struct Operand {
    const half_t* ptr;
    int64_t ld;
    int64_t batch_stride;
};

struct GemmShape {
    int M, N, K;        // multiples of the tile sizes / 64
    int k_split;        // grid.y
    int k_chunk;        // K range per split, multiple of 64
    int sym;            // 1: only upper-triangular tiles, mirrored on store
};

// out = mul^p * (ca * acc + cs * src), stored as fp16; optional mirror for
// symmetric results and optional per-tile sum of squares of the output.
struct EpiAffine {
    half_t* out; int64_t ld_out; int64_t stride_out;
    const half_t* src; int64_t ld_src; int64_t stride_src;
    const float* mul; int mul_pow;      // per-matrix factor mul[z]^mul_pow
    float ca, cs;
    float* sumsq;                       // [z][tile] partial sums, or null
    int tiles_per_mat;
};

// fp32 partial products of one K split: out[z][split][mm][nn]
struct EpiPartial {
    float* out; int64_t ld_out; int64_t stride_split; int64_t stride_mat;
};

// NormPre-L apply: T = Psi + acc in the W layout, then the RMS-matched
// weight update W <- W - lr (s T + wd W) with s = rms sqrt(mn) / ||T||_F.
struct EpiApplyUpdate {
    const half_t* psi; int64_t ld_psi; int64_t stride_psi;
    const float* tnorm2;                // per matrix ||T||_F^2 (from the norm pass)
    int rows, cols;                     // real sizes of W
    float lr, wd, target_rms;
    int vec_ok;                         // W rows 16-byte aligned (cols % 4 == 0)
    PtrChunk ptrs;                      // w[] used
};

// NormPre-L norm pass: the same T = Psi + acc, reduced to per-tile partial
// sums of T^2 over the real rows x cols region (no write of T or W).
struct EpiApplyNorm {
    const half_t* psi; int64_t ld_psi; int64_t stride_psi;
    int rows, cols;
    float* sumsq; int tiles_per_mat;
    const int* need;                    // if set: only matrices with need[z] != 0
};

enum class EpiKind { Affine, Partial, Apply, ApplyNorm };

// Launchers (gemm kernels, np_gemm.hip).  `layout` selects which operands
// are MN-major: 0 = both K-major, 1 = B MN-major, 2 = both MN-major.
// Skinny64 / Skinny64W / Skinny128: split-K sketch products, l-major rows
// of 64 (or 128) by 256 (or 512) output columns.
enum class TileCfg { Big, Big256, Skinny64, Skinny64W, Skinny128, Apply };
hipError_t launch_gemm_affine(TileCfg cfg, int layout, Operand A, Operand B,
                              GemmShape sh, int batch, const EpiAffine& e,
                              hipStream_t s);
hipError_t launch_gemm_partial(TileCfg cfg, int layout, Operand A, Operand B,
                               GemmShape sh, int batch, const EpiPartial& e,
                               hipStream_t s);
// Split-K sketch products of several shape groups with one padded width l
// (M) in one launch.  Group g covers launch matrices [zbeg[g], zbeg[g + 1]):
// operands a (M x K, K-major) and b (the W-layout Psi, per-matrix strides),
// output length N, reduction length K in `splits` chunks of k_chunk, fp32
// partials out[i][split][mm][nn] (ld N).  N, K and k_chunk are multiples of
// the tile sizes and of 64; chunk `splits - 1` is the last non-empty one.
// A group with one split and a final output (out32 and/or out16 set) gets
// the product itself instead of a partial: fp32 into out32 and fp16 of
// scale16 times it into out16 (ld N, matrix stride stride_out), the values a
// one-split reduction would write.
struct SketchGroups {
    int n;
    int zbeg[kMaxItems + 1];
    const half_t* a[kMaxItems]; int64_t lda[kMaxItems]; int64_t a_stride[kMaxItems];
    const half_t* b[kMaxItems]; int64_t ldb[kMaxItems]; int64_t b_stride[kMaxItems];
    int N[kMaxItems], K[kMaxItems], k_chunk[kMaxItems], splits[kMaxItems];
    float* out[kMaxItems]; int64_t stride_split[kMaxItems]; int64_t stride_mat[kMaxItems];
    float* out32[kMaxItems]; half_t* out16[kMaxItems]; float scale16[kMaxItems]; int64_t stride_out[kMaxItems];
};
hipError_t launch_gemm_partial_grouped(TileCfg cfg, int layout, int M, const SketchGroups& g, hipStream_t s);
// Newton-Schulz combines X <- a X + B X of the wide shape groups of one s in
// one launch (B MN-major: the layout-1 combine).  Group g covers launch
// matrices [zbeg[g], zbeg[g + 1]) with its own B (s x s), X (s x N), output,
// source, first-iteration scale (mul[2 i]; null = 1) and per-tile sums of
// squares (sumsq, tiles per matrix; null = none).  ca, cs and mul_pow come
// from the EpiAffine argument.
struct CombineGroups {
    int n;
    int zbeg[kMaxItems + 1];
    const half_t* a[kMaxItems]; int64_t lda[kMaxItems]; int64_t a_stride[kMaxItems];
    const half_t* b[kMaxItems]; int64_t ldb[kMaxItems]; int64_t b_stride[kMaxItems];
    int N[kMaxItems];
    half_t* out[kMaxItems]; int64_t ld_out[kMaxItems]; int64_t stride_out[kMaxItems];
    const half_t* src[kMaxItems]; int64_t ld_src[kMaxItems]; int64_t stride_src[kMaxItems];
    const float* mul[kMaxItems];
    float* sumsq[kMaxItems]; int tiles[kMaxItems];
};
hipError_t launch_gemm_combine_grouped(TileCfg cfg, int s_dim, const CombineGroups& g, const EpiAffine& e,
                                       hipStream_t s);
hipError_t launch_gemm_apply(Operand A, Operand B, GemmShape sh, int batch,
                             const EpiApplyUpdate& e, hipStream_t s);
hipError_t launch_gemm_apply_norm(Operand A, Operand B, GemmShape sh, int batch,
                                  const EpiApplyNorm& e, hipStream_t s);
// Grouped symmetric Gram (X X^T with layout 0, Y^T Y with layout 2): shape
// groups of one s (same padded s x s output) in one launch.  Group g covers
// launch matrices [zbeg[g], zbeg[g + 1]) with its own operand (ld,
// per-matrix stride), K and
// first-iteration scale (mul[2 i], squared; null = 1); its matrices land at
// output indices zout[g] + i.
constexpr int kMaxGramGroups = 6;
struct GramGroups {
    int n;
    int zbeg[kMaxGramGroups + 1];
    const half_t* x[kMaxGramGroups];
    int64_t ld[kMaxGramGroups];
    int64_t stride[kMaxGramGroups];
    int K[kMaxGramGroups];
    const float* mul[kMaxGramGroups];
    int zout[kMaxGramGroups];
};
hipError_t launch_gemm_gram_grouped(TileCfg cfg, int layout, const GramGroups& g, int sp, const EpiAffine& e,
                                    hipStream_t s);
int gemm_tile_m(TileCfg cfg);
// Kernel timing hand-off (instrumented steps only): while a start/stop event
// pair is armed on this thread, the next GEMM launch records it at its own
// start and end (hipExtLaunchKernelGGL) and disarms it.
void arm_launch_events(hipEvent_t start, hipEvent_t stop);
bool disarm_launch_events();        // true if the pair was still armed

int gemm_tile_n(TileCfg cfg);

// ------------------------------------------------- elementwise kernels ---
// Momentum + relaxed tangent + diagonal-Gram normalization.
struct NormArgs {
    PtrChunk ptrs;
    int rows, cols;                 // real W sizes
    int64_t ld_psi;                 // padded row length of the Psi workspace
    int64_t rows_pad;               // padded row count of the Psi workspace
    half_t* psi; int64_t stride_psi;   // fp16 Psi, W layout, zero padded
    float* psi32; int64_t stride_psi32; // optional fp32 copy (debug), ld = cols
    float* psisq; int64_t stride_psisq; // per active row ||psi_i||^2
    float mu, eps;
    int vec_ok;                     // 16-byte aligned W, M, G rows
    int tangent;                    // kTangentRelaxed / kTangentNone / kTangentStrict
    float* xsq;                     // optional per active row ||x_i||^2 (stride_psisq)
    // Finite check: non-finite G and M_prev entries count as zero in M,
    // non-finite W entries as zero in the tangent; the number of non-finite
    // G, M_prev and W entries per row (row-active) or per stats block
    // (column-active) goes to nfin[z * stride_nfin + slot].
    int* nfin; int64_t stride_nfin;
};
constexpr int kTangentRelaxed = 0, kTangentNone = 1, kTangentStrict = 2;
// Slots of non-finite counts a normalization launch writes per matrix.
int64_t nonfinite_slots(const NormArgs& a, bool row_active, int row_chunk);
// status[idx[i]] = sum of the matrix's count slots (i < count <= kChunk).
struct IdxChunk { int idx[kChunk]; };
hipError_t launch_count_reduce(const int* nfin, int64_t slots, int64_t stride, const IdxChunk& idx, int count,
                               long long* status, hipStream_t s);
hipError_t launch_normalize_rows(const NormArgs& a, int batch, hipStream_t s);
// Column-active orientation: one pass where a strip of SW columns of M and
// W fits the registers of one block (cols_fused_width(a) = SW, padded
// columns of at most 2048 rows, 16-byte aligned rows), else a statistics
// pass and a normalize pass over `partials`.
int cols_fused_width(const NormArgs& a);
hipError_t launch_normalize_cols(const NormArgs& a, int batch, double* partials,
                                 int row_chunk, hipStream_t s);
int64_t normalize_cols_partials(int rows, int cols_pad, int row_chunk);
// Both-axes normalization, second half: every column of the fp16 Psi (and of
// the fp32 debug copy) scaled to unit norm, zero columns kept at zero; the
// squared column norms go to psisq.  `part` holds part_floats floats per
// matrix (row-chunk partial sums, then the column factors).
// X_s = sqrt(a / tot) D Psi over the padded W layout (zero padding kept):
// D = diag(||x_i||) of the active rows (rows for k = 0, columns for k = 1),
// tot = xtot[2 z + 1] = ||X||_F^2.
hipError_t launch_source_x(const half_t* psi, int64_t ld, int64_t stride, int rows, int cols, int rows_pad, int k,
                           int active, const float* xsq, int64_t stride_xsq, const float* xtot, half_t* xs,
                           int batch, hipStream_t s);
hipError_t launch_psi_col_normalize(const NormArgs& a, int batch, float* part, int64_t part_floats, int row_chunk,
                                    hipStream_t s);

// out[z] = sum_i in[z*n + i] in a fixed order (per-matrix ||T||_F^2 from
// per-tile partial sums); with `need`, only for the matrices with
// need[z] != 0.
hipError_t launch_sum_partials(const float* in, int n, float* out, int batch, hipStream_t s,
                               const int* need = nullptr);
// NormPre-L ||T||_F^2 in closed form (App. B), for several shape groups in
// one launch: matrix z of the launch is matrix z - zbeg[g] of group g.  With
// the selected Ritz values the first nsel[i] of the descending list ritz[i]
// (stride ritz_stride), ||T||_F^2 = ||Psi||_F^2 - sum_C (lambda_i - 1),
// psi2[i * 2] being ||Psi||_F^2.  It is written to tn2[i] unless the selected
// modes hold more than `frac` of ||Psi||_F^2 (or the result is not
// positive); need[i] = 1 marks those matrices, whose norm the norm pass over
// T supplies instead.
struct LNormGroups {
    int n;
    int zbeg[kMaxItems + 1];
    const float* psi2[kMaxItems];
    const float* ritz[kMaxItems]; int64_t ritz_stride[kMaxItems];
    const int* nsel[kMaxItems];
    float* tn2[kMaxItems];
    int* need[kMaxItems];
    float frac;
};
hipError_t launch_l_norm_closed(const LNormGroups& g, hipStream_t s);

// Per-matrix Newton-Schulz pre-scale c = 1 / (sqrt(sum psisq) + eps) and
// ||Psi||_F^2: out[z*2] = c, out[z*2+1] = ||Psi||^2.
hipError_t launch_psi_scale(const float* psisq, int64_t stride, int active_rows,
                            float eps, float* out, int batch, hipStream_t s);

// NormPre-G final step: ||T||^2 from per-tile partial sums, then
// W <- W - lr (rms sqrt(mn) T / ||T|| + wd W).
struct GUpdateArgs {
    PtrChunk ptrs;
    int rows, cols;
    const half_t* t; int64_t ld_t; int64_t stride_t;
    const float* tnorm2;            // ||T||_F^2 of matrix z at tnorm2[z * tnorm2_stride]
    int64_t tnorm2_stride;
    float fixed_scale;              // > 0: U = fixed_scale * T instead of the RMS match
    float lr, wd, target_rms;
    float* t32; int64_t stride_t32; // optional fp32 copy of T (debug)
    int vec_ok;                     // 16-byte aligned W rows
};
hipError_t launch_g_update(const GUpdateArgs& a, int batch, hipStream_t s);
// Muon input: momentum update with per-block sums of M^2 (part, one float per
// block, momentum_sumsq_blocks(rows*cols) blocks), then X0 = M * scale[2z]
// to fp16 in the zero-padded workspace.
int momentum_sumsq_blocks(int64_t elems);
hipError_t launch_momentum_sumsq(const NormArgs& a, int batch, float* part, int64_t stride_part, hipStream_t s);
hipError_t launch_scaled_cast(const NormArgs& a, int batch, const float* scale, hipStream_t s);

// ------------------------------------------------------ sketch kernels ---
// Omega^T (l x b) in fp16, zero padded to (l_pad x b_pad), ld = b_pad.
struct OmegaArgs {
    uint64_t seed; int64_t step;
    int ids[kChunk];            // matrix id (index in the caller's list)
    int b, ell, ell_pad; int64_t ld;
    half_t* out; int64_t stride;
};
hipError_t launch_omega_f16(const OmegaArgs& a, int batch, hipStream_t s);
hipError_t launch_omega_f32(uint64_t seed, int64_t step, int id, int64_t b,
                            int ell, float* out, hipStream_t s);

// Sum of K-split partials -> fp32 (l_pad x len) and scaled fp16 copy.
hipError_t launch_reduce_splits(const float* part, int splits, int64_t stride_split,
                                int64_t stride_mat, int rows, int64_t len,
                                float* out32, half_t* out16, float scale16,
                                int64_t stride_out, int batch, hipStream_t s);
// The split sums of several sketch products in one launch: group g covers
// launch matrices [zbeg[g], zbeg[g + 1]) with its own partials and outputs
// (arguments as in launch_reduce_splits; rows x len per matrix).
struct ReduceGroups {
    int n;
    int zbeg[kMaxItems + 1];
    const float* part[kMaxItems];
    int splits[kMaxItems];
    int64_t stride_split[kMaxItems], stride_mat[kMaxItems];
    int64_t n4[kMaxItems];                       // rows * len / 4
    float* out32[kMaxItems];
    half_t* out16[kMaxItems];
    float scale16[kMaxItems];
    int64_t stride_out[kMaxItems];
};
hipError_t launch_reduce_splits_grouped(const ReduceGroups& g, hipStream_t s);

// Fixed number of length-chunk slots of the fp64 Gram partial sums (unused
// slots hold zeros); its consumers always add all of them.
constexpr int kGramChunks = 16;

// fp64 Gram of the rows of l-major fp32 matrices V (l_pad x len each):
// partial[z][chunk][c][d] = sum_{j in chunk} V[c][j] V[d][j], upper tiles.
// Every launch writes all kGramChunks chunk slots of chunk_len (slots past
// len hold zeros).
struct Gram64Items {
    int n;
    int ell;                                     // rows of each matrix that enter the Gram
    int zbeg[kMaxItems + 1];
    const float* v[kMaxItems];
    int64_t ld[kMaxItems];
    int64_t stride[kMaxItems];
    int64_t len[kMaxItems];
    int chunk_len[kMaxItems];
};
hipError_t launch_gram64(const Gram64Items& t, int ell_pad, double* partial, hipStream_t s);
// Element (c, d) of the summed Gram (full symmetric view of the upper 64 x 64
// tiles gram64 writes): the kGramChunks partial sums are all requested
// before any is added, so one memory latency covers the element; they are
// added in chunk order.
__device__ __forceinline__ double gram_at(const double* p, int ell_pad, int c, int d) {
    if ((c >> 6) > (d >> 6)) { const int t = c; c = d; d = t; }
    const double* q = p + (int64_t)c * ell_pad + d;
    const int64_t cs = (int64_t)ell_pad * ell_pad;
    double v[kGramChunks];
#pragma unroll
    for (int k = 0; k < kGramChunks; ++k) v[k] = q[k * cs];
    double s = 0.0;
#pragma unroll
    for (int k = 0; k < kGramChunks; ++k) s += v[k];
    return s;
}
int gram64_chunks(int64_t len, int chunk_len);

// Cholesky (with dropping of numerically dependent columns) of the summed
// Gram, then R^{-1}; writes fp32 Rinv (l_pad x l_pad, zero padded).
hipError_t launch_chol_inv(const double* partial, int chunks, int ell, int ell_pad,
                           double* scratch, float* rinv, int batch, hipStream_t s);

// out = M^T V  (M: l_pad x l_pad fp32, V: l_pad x len fp32, l-major),
// optional outputs: fp32 l-major, fp16 l-major, fp16 len-major (len x l_pad).
struct SmallMulItem {
    const float* mat;                            // first matrix's M; stride l_pad^2
    const float* v; int64_t ld_v; int64_t stride_v;
    int64_t len, len_pad;
    float* out32; int64_t stride_out32;          // ld = ld_v
    half_t* out16; int64_t stride_out16;         // ld = ld_v
    half_t* out16t; int64_t stride_out16t;       // ld = ell_pad
};
struct SmallMulArgs {
    int ell, ell_pad;
    int n;
    int zbeg[kMaxItems + 1];
    SmallMulItem it[kMaxItems];
};
hipError_t launch_small_mul(const SmallMulArgs& a, hipStream_t s);

// Jacobi eigensolver of Gamma_Q (summed fp64 partials), selection of the
// top-min(r, l) Ritz values > 1, K = Z_C diag(lambda^-1/2 - 1) Z_C^T (fp32,
// l_pad x l_pad).
struct EigArgs {
    const double* partial; int chunks;
    int ell, ell_pad, rank;
    float* scratch;             // 2 * l_pad * l_pad floats per matrix
    float* kmat;                // l_pad x l_pad per matrix
    float* ritz; int ritz_stride;
    int* nsel;
    int max_sweeps;
};
hipError_t launch_eig_select(const EigArgs& a, int batch, hipStream_t s);

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t s);

// Streaming ceilings with the byte mixes of the normalization passes (n
// elements, a multiple of 4; 16-byte aligned buffers):
//   0: read a, b, c, write o32 = 0.95 a + b and o16 = fp16(c)   18 B/element
//   1: read a, b, c, write o32 = 0.95 a + b + c                16 B/element
//   2: read a, b, write o16 = fp16(a - b)                     10 B/element
//   3: read a, write o32 = a                                    8 B/element
hipError_t launch_stream_probe(int mix, int64_t n, const float* a, const float* b, const float* c, float* o32,
                               half_t* o16, hipStream_t s);

// Descent alignment (App. A, training dynamics): per matrix the cosine of the
// gradient G and the update direction Phi = (W_before - W_after) / lr -
// wd W_before (the update before learning-rate scaling, weight decay
// excluded).  Partial sums per block (fp64), then one block reduces them in
// a fixed order to cos[z] and their mean.
struct AlignChunk {
    const float* g[kChunk];
    const float* wb[kChunk];
    const float* wa[kChunk];
    int64_t n[kChunk];
};
constexpr int kAlignBlocks = 128;
hipError_t launch_alignment_partials(const AlignChunk& c, int cnt, double lr, double wd, double* part,
                                     hipStream_t s);
hipError_t launch_alignment_finalize(const double* part, int num_mats, double* cos_out, double* mean_out,
                                     hipStream_t s);
// Q <- Q + a I in place for `count` contiguous sp x sp fp16 matrices.
hipError_t launch_add_diag(half_t* q, int64_t sp, int count, float a, hipStream_t s);

// ------------------------------------------ dense symmetric eigensolver ---
// Workspace of one launch of matrices of equal order n (per matrix: A n x n
// fp32, vec 4 n, d / e / tau n each; per matrix and requested eigenvector:
// lu 5 n, y n; fp64 unless stated).
struct TriWork {
    float* A;       // the matrix on entry; reflectors in its rows on exit
    double* vec;
    double* d;
    double* e;
    double* tau;
    double* lu;     // inverse iteration: 6 n doubles per eigenvector
    double* y;
};
// Symmetrized copy of the leading n x n block of an fp32 matrix (ld ldg).
hipError_t launch_gamma_sym(const float* g, int64_t ldg, int64_t strideg, int n, float* A, int batch,
                            hipStream_t s);
// Householder reduction of A to tridiagonal form (d, e), reflectors kept.
hipError_t launch_tridiagonalize(const TriWork& w, int n, int batch, hipStream_t s);
// Eigenvalues first .. first + nvals - 1 in descending order (0 = largest).
hipError_t launch_tri_eigvals(const TriWork& w, int n, int first, int nvals, double* out, int64_t stride_out,
                              int batch, hipStream_t s);
// Unit eigenvectors of A for the given eigenvalues (nvals per matrix,
// descending), as fp32 rows of out (ld_out >= n, zero padded; rows nvals ..
// rows_out - 1 zero).
hipError_t launch_tri_eigvecs(const TriWork& w, int n, const double* lam, int nvals, float* out, int64_t ld_out,
                              int rows_out, int64_t stride_out, int batch, hipStream_t s);
// Ritz pairs through the dense eigensolver (for l above the Jacobi kernels'
// sweet spot): Gamma_Q from the summed fp64 Gram partials, its top
// min(r, l) eigenpairs, the selection lambda > 1 and K = Z_C diag(lambda^-1/2
// - 1) Z_C^T, with the outputs of launch_eig_select.  zbuf: top x l floats
// per matrix; lam: top doubles per matrix.
hipError_t launch_eig_select_dense(const EigArgs& a, const TriWork& w, double* lam, float* zbuf, int batch,
                                   hipStream_t s);
// Gamma = Psi Psi^T (layout 0) or Psi^T Psi (layout 2) in fp32, full tiles.
hipError_t launch_gemm_gram_f32(int layout, Operand A, Operand B, GemmShape sh, int batch, const EpiPartial& e,
                                hipStream_t s);

}  // namespace np
