// Launch interface of the gfx950 kernels (host side).  Each launcher queues work on
// the given stream and returns the launch status; argument validation is the
// caller's job (the C-ABI layer checks every shape before calling in here).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/jolt.h"

// ----------------------------------------------------------------- residual calibration
struct Eps2Args {
  uint64_t seed;
  int64_t n_samples;
  int32_t group;
  float inv_sqrt_d;
  double *partials;         // [blocks][4]
};


// ----------------------------------------------------------------- fused reconstruction
// X~_s rebuilt on the fp16 matrix cores inside the residual / decode passes: for fp16
// factors as 2^e_s (U^_T G^_s) U^_d^T (launch_core_prepare), for fp32 factors as U^_T W_s.
struct FusedCell {
  const void *UT;           // blob U_T section: T x rT, fp16 or fp32 (the call's factor type)
  float *Wt;                // m slices of d x ldw floats.  fp32 factors: W_s^T = 2^e_s U^_d G^_s^T,
                            // which launch_w_prepare rewrites in place, entry by entry, as the
                            // fp16 pair (hi, lo) of W_s^T 2^-k_s (hi in the low half-word).
                            // fp16 factors: G^_s^T as fp16, round32(r_d) rows of round16(r_T)
                            // (launch_core_prepare)
  int32_t *wexp;            // m per-slice exponents: k_s of W_s, or ky_s of Y_s = U^_T G^_s
  const uint16_t *G;        // blob core section (m x rT x rd fp16) and its per-slice exponents
  const int8_t *gexp;
  const uint16_t *Ud;       // blob U_d section (d x rd fp16)
  uint16_t *udp;            // d x round32(rd): U^_d with columns in the fused kernel's slot order
  const void *x;            // residual: cache cell base (strided, input type)
  void *out;                // decode: output cell base (strided, output type)
  uint8_t *codes;           // packed codes (written by the residual pass, read by decode)
  uint16_t *scales;         // fp16 group scales
  float *xt_out;            // export: X~ (m x T x d fp32, contiguous)
  int32_t rT, bits, ldw, rd;
};
enum { FUSED_RESIDUAL = 0, FUSED_DECODE = 1, FUSED_XTILDE = 2 };
struct FusedArgs {
  const FusedCell *cells;   // device [n_cells]
  const float *signs;       // device [n_cells][d]
  int32_t n_cells, m, T, heads, group;
  int32_t tiles_t, total, per_xcd;    // set by launch_fused
  int64_t s_layer, s_head, s_tok;     // cell strides (input for the residual, output for decode)
  float inv_sqrt_d;
  int32_t rope, rope_offset, pad;
  double rope_log2_base;
};
int fused_tile_tokens();
// Per (cell, slice): k_s = the smallest power of two with max |W_s| 2^-k_s <= 2^14, then
// every entry of W_s^T rewritten in place as its fp16 hi + lo split (zeros past r_T).
hipError_t launch_w_prepare(const FusedCell *cells_dev, int n_cells, int m, int d, hipStream_t st);
// fp16 factors: per (cell, slice) G^_s^T zero-padded into the slice's W area and the exponent
// ky_s with |U^_T G^_s| 2^-ky_s <= 2^15; per cell the permuted copy udp of U^_d with the
// rotation signs (device [n_cells][d]) folded into its rows.
hipError_t launch_core_prepare(const FusedCell *cells_dev, const float *signs_dev, int n_cells, int m, int d,
                               hipStream_t st);
// io_dtype: the cache type (residual) or the output type (decode); split_factors: the
// factors are fp32 (U_T split into two fp16 terms)
hipError_t launch_fused(FusedArgs a, int mode, int d, int io_dtype, bool split_factors, hipStream_t st);
hipError_t launch_rotation_signs(const uint64_t *seeds_dev, int n_cells, int d, float *signs,
                                 hipStream_t st);
int eps2_blocks();
hipError_t launch_eps2_partial(const Eps2Args &a, int d, hipStream_t st);

// ----------------------------------------------------------------- generic MFMA GEMM
// C[b] = alpha * op(A[b]) op(B[b]) + beta * C[b] for a table of problems b.
// An operand is a 2-D view with element (row, col) at
//   ptr + seg_off(col / seg_len) + row * ld + (col % seg_len)
// where seg_off(s) = (s / seg_heads) * seg_hi + (s % seg_heads) * seg_lo (no segmentation
// when seg_len = 0).  A is M x K: "k-contiguous" (row = m, col = k) or
// "m-contiguous" (row = k, col = m).  B is K x N: "k-contiguous" (row = n, col = k)
// or "n-contiguous" (row = k, col = n).
enum GemmType { GT_BF16 = 0, GT_F16 = 1, GT_F32 = 2, GT_F64 = 3 };

// Element (row, col) of an operand sits at row * ld + col, or, when seg_len > 0, the
// contiguous index col runs over segments of seg_len elements (seg_len a power of two):
// segment s = col / seg_len starts at (s / seg_heads) * seg_hi + (s % seg_heads) * seg_lo.
// seg_shift = log2(seg_len) and heads_magic = ceil(2^32 / seg_heads) make both divisions
// a shift and a multiply (exact for s < 2^20, seg_heads < 2^12); build with seg_operand().
struct GemmOperand {
  const void *ptr;
  int64_t ld;
  int64_t seg_hi, seg_lo;
  int32_t seg_len, seg_heads;
  int32_t seg_shift, pad_;
  uint64_t heads_magic;
};

inline GemmOperand seg_operand(const void *ptr, int64_t ld, int64_t seg_hi, int64_t seg_lo,
                               int32_t seg_len, int32_t seg_heads) {
  GemmOperand o{ptr, ld, seg_hi, seg_lo, seg_len, seg_heads, 0, 0, 0};
  if (seg_len > 0) {
    while ((1 << o.seg_shift) < seg_len) ++o.seg_shift;
    o.heads_magic = ((uint64_t(1) << 32) + (uint64_t)seg_heads - 1) / (uint64_t)seg_heads;
  }
  return o;
}

__device__ __forceinline__ int64_t operand_col(const GemmOperand &op, int col) {
  if (op.seg_len == 0) return col;
  const uint32_t s = (uint32_t)col >> op.seg_shift;
  const uint32_t hq = (uint32_t)(((uint64_t)s * op.heads_magic) >> 32);
  const uint32_t hr = s - hq * (uint32_t)op.seg_heads;
  return (int64_t)hq * op.seg_hi + (int64_t)hr * op.seg_lo + (col & (op.seg_len - 1));
}

struct GemmProblem {
  GemmOperand A, B;
  float *C;              // fp32 output (row-major M x N with ldc)
  int64_t ldc;
  int32_t M, N, K;
  float alpha, beta;
  int32_t lower_only;    // compute only tiles with tile_m >= tile_n (symmetric outputs)
  int32_t c_trans;       // bf16 kernel only: store element (m, n) at C[n * ldc + m]
  const int8_t *alpha_exp2;  // optional: alpha is multiplied by 2^(*alpha_exp2)
};

// fp32 MFMA GEMM (mode 1): A/B of types ta/tb (bf16, fp16 or fp32) converted exactly to
// fp32; every table accepted.
hipError_t launch_gemm(const GemmProblem *probs_dev, int n_probs, int max_M, int max_N,
                       int mode, int ta, int tb, bool a_kcontig, bool b_kcontig, hipStream_t st);
// bf16 matrix-core GEMM; ta/tb GT_BF16 (used as is) or GT_F32 (split into bf16 hi + lo).
// gemm16_prepare() runs on the host copy of the table before it is uploaded: it returns
// false when a layout condition of the kernel is not met (use launch_gemm then), and may
// rewrite the table and the type / layout arguments (an fp32 A is moved to the B side by
// computing C^T) and picks the tile height bm for launch_gemm16.
// tile code of launch_gemm16 besides the row counts 128 and 256: 256 x 256 tiles
constexpr int GEMM16_SQUARE256 = 512;
bool gemm16_prepare(GemmProblem *probs_host, int n_probs, int &ta, int &tb, bool &a_kcontig,
                    bool &b_kcontig, int &bm);
// C = alpha A B + beta C over the lower tiles for fp32 A, B stored mn-contiguous, K <= 64,
// on the bf16 matrix cores with each operand split into three bf16 terms (fp32-level
// accuracy): the rank-2k update of the blocked tridiagonalisation.
hipError_t launch_update3(const GemmProblem *probs_dev, int n_probs, int max_MN, hipStream_t st);
hipError_t launch_gemm16(const GemmProblem *probs_dev, int n_probs, int max_M, int max_N, int ta,
                         int tb, bool a_kcontig, bool b_kcontig, int bm, bool lower_only,
                         hipStream_t st);

// ----------------------------------------------------------------- feature Gram / energy
// F[cell] = sum over rows of x^T x for the row set {(s, r) : s < nseg, r < rows_per_seg}
// with row (s, r) at base + seg_off(s) + r * row_stride; also sum x^2 (fp64) and a
// non-finite flag.  Partials are reduced by launch_feature_gram_reduce.
struct FGramCell {
  const void *base;
  int32_t rows_per_seg;     // rows of each segment for this cell
  int32_t pad;
};
struct FGramArgs {
  const FGramCell *cells;
  int32_t n_cells, nseg, seg_heads;
  int64_t seg_hi, seg_lo, row_stride;
  int32_t chunks_per_cell;  // work items per cell (each a contiguous run of rows)
  int32_t vec16;            // set by the caller: every row start is 16-byte aligned
  float *partial_F;         // [n_cells][chunks][d][d]
  double *partial_E;        // [n_cells][chunks]
  int32_t *nonfinite;       // [n_cells]
};
hipError_t launch_feature_gram(const FGramArgs &a, int d, int dtype, hipStream_t st);
// F_out[cell] (fp32, d x d) and E_out[cell] (fp64) from the partials
hipError_t launch_feature_gram_reduce(const FGramArgs &a, int d, float *F_out, double *E_out,
                                      hipStream_t st);

// Running sums over the n_k matrices of each cell, in place: M[c][k] <- sum_{j <= k} M[c][j]
// (elems floats per matrix, fp64 accumulation, fp32 stores).
hipError_t launch_prefix_sum_mats(float *M, int n_cells, int n_k, int64_t elems, hipStream_t st);

// ----------------------------------------------------------------- slice-mode Gram
// S[cell][s][s'] = sum over tokens t and features f of X[s][t][f] X[s'][t][f] (the Gram of
// the slice unfolding: appendix A's head mode).  Workgroup (pair of 16-slice tiles, token
// chunk, cell) writes an fp64 partial for its tile pair; the reduce adds the chunks in a
// fixed order and writes the full symmetric fp32 matrix.
struct SliceGramArgs {
  const FGramCell *cells;   // base per cell
  int32_t n_cells, m, T, heads;
  int64_t s_layer, s_head, s_tok;
  int32_t tiles, chunks;    // ceil(m / 16) slice tiles; token chunks per cell
  double *partial;          // [n_cells][chunks][m][m]
};
hipError_t launch_slice_gram(const SliceGramArgs &a, int d, int dtype, hipStream_t st);
hipError_t launch_slice_gram_reduce(const SliceGramArgs &a, float *S_out, hipStream_t st);

// ----------------------------------------------------------------- attention on the factors
// One item = a layer of a compressed key cell and of the matching value cell, and n_q
// query heads; key-value head h of the layer is slice s = layer * heads + h, query head j
// reads head j / (n_q / heads).
struct AttnBlob {
  const void *UT, *Ud, *G;     // fp16 (f16 = 1) or fp32 factors: T x rT, d x rd, m x rT x rd
  const int8_t *gexp;          // per-slice core exponents
  const uint8_t *codes;        // packed residual codes (s, t, f) order, LSB first
  const uint16_t *scales;      // fp16 group scales
  int32_t rT, rd, bits, f16;
};
struct AttnItem {
  AttnBlob k, v;
  int32_t layer, pad;
};
struct AttnArgs {
  const AttnItem *items;
  const float *signs;          // [n_items][2][d]: key, value rotation signs
  const float *Q;              // [n_items][n_q][d]
  float *O;                    // [n_items][n_q][d]
  float *gk;                   // [n_items][n_q][rk_max]: 2^e G_s U_d^T q (key side)
  float *qr;                   // [n_items][n_q][d]: H (signs . q) / sqrt(d)
  float *part;                 // [n_items][chunks][n_q][2 + rv_max + d] chunk partials
  int32_t n_items, n_q, heads, T, group, chunks, rk_max, rv_max;
  float scale, inv_sqrt_d;
};
constexpr int ATTN_CHUNK = 64;      // tokens per workgroup of the chunk pass
constexpr int ATTN_QMAX = 64;       // query heads per item
constexpr int ATTN_REP_MAX = 8;     // query heads per key-value head
constexpr int ATTN_RT_MAX = 1024;   // largest value rank the combine kernel stages in LDS
hipError_t launch_attend(const AttnArgs &a, int d, hipStream_t st);
// fixed per-device scratch of the allocation-free attention entry point
constexpr size_t ATTN_SCRATCH_BYTES = JOLT_ATTEND_SCRATCH_BYTES;
constexpr int ATTN_SCRATCH_DEVICES = 64;
// the calling thread must have `device` current
hipError_t attend_scratch_address(int device, void **ptr);

// ----------------------------------------------------------------- eigensolver
struct EigBatch {
  float *A;              // [n_mat][n][n] row-major; lower triangle read, overwritten with
                         // the Householder vectors
  int64_t mat_stride;    // elements between matrices
  int32_t n_mat, n;
  double *d, *e;         // tridiagonal [n_mat][n]
  float *tau;            // [n_mat][n]
  double *lam;           // eigenvalues, descending [n_mat][n]
  int32_t refl_off;      // row of reflector i's unit is i + refl_off (0 read as 1: one-stage)
  int32_t pad_;
};
inline __host__ __device__ int refl_off(const EigBatch &b) { return b.refl_off > 0 ? b.refl_off : 1; }
// Householder tridiagonalisation (lower): small n in one workgroup per matrix.
hipError_t launch_sytrd_small(const EigBatch &b, hipStream_t st);
// Blocked multi-workgroup tridiagonalisation for large n (panels of nb columns).
// work: sytrd_large_work_floats() device floats; tables: sytrd_large_table_entries().
struct SytrdArgs {
  float *A;
  int64_t mat_stride;
  int32_t n, nb, slots, pad;
  double *d, *e;
  float *tau;
  float *work;           // per-matrix panels, vectors and partial sums
  int64_t work_stride;   // floats between matrices in work
};
size_t sytrd_large_work_floats(int n_mat, int n, int nb);
size_t sytrd_large_table_entries(int n_mat, int n, int nb);
// host-side GEMM table of the panel updates (sytrd_large_table_entries() entries); the
// launch sequence itself is fixed for a given shape and pointers (it may be captured once
// into a graph and replayed).
void sytrd_large_tables(const EigBatch &b, float *work, int nb, GemmProblem *tab_host);
hipError_t launch_sytrd_large(const EigBatch &b, float *work, int nb, const GemmProblem *tab_dev,
                              hipStream_t st, int m0 = 0, int m1 = -1);
// all eigenvalues of the tridiagonal (fp64 bisection), descending
hipError_t launch_tridiag_eigvals(const EigBatch &b, hipStream_t st);
// top-k eigenvectors of the tridiagonal by fp64 inverse iteration, orthogonalised
// within clusters; Z [n_mat][n][kmax] fp64 row-major (ldz = kmax); k per matrix.
struct InvitWork {
  double *Z;             // [n_mat][n][ldz]
  double *lu;            // scratch [n_mat][3][n][ldlu], columns processed ldlu at a time
  int32_t ldz, ldlu;
  const int32_t *k;      // device [n_mat] vectors wanted per matrix
  int32_t *status;       // device [n_mat], zeroed by the launcher: set to 1 when a vector's
                         // solution growth misses the convergence bound
  int32_t iters;         // inverse-iteration sweeps per vector (normally 2)
  int32_t pad;
};
hipError_t launch_tridiag_eigvecs(const EigBatch &b, const InvitWork &w, int kmax,
                                  hipStream_t st);
// U = Q Z for the Householder vectors stored in A (Q = H_0 ... H_{n-2}), blocked into
// panels of backtransform_nb() reflectors applied as I - V T V^T with GEMMs.  U fp32
// [n_mat] x (n x ldu) at u_stride, first k[mat] columns written (k_host: the host copy of
// the per-matrix counts; each matrix's products run over its own k[mat] columns).  Needs
// backtransform_scratch_floats() device floats and backtransform_table_entries()
// GemmProblem slots on device (tab_dev) and host (tab_host).
int backtransform_nb();
size_t backtransform_scratch_floats(int n_mat, int n, int kmax);
size_t backtransform_table_entries(int n_mat, int n);
// u_ready: U already holds the vectors to transform (fp32), Z is not read.
hipError_t launch_backtransform(const EigBatch &b, const InvitWork &w, int kmax, const int *k_host, float *U,
                                int64_t ldu, int64_t u_stride, float *scratch, GemmProblem *tab_dev,
                                GemmProblem *tab_host, hipStream_t st, bool u_ready = false);

// Two-stage tridiagonalisation for large n (k_sb.hip): dense to band of half-bandwidth
// sb_band() by panel QR and rank-2 sb_band() updates, then band to tridiagonal by bulge
// chasing.  Leaves d, e, tau and the stage-1 reflectors in A (explicit, unit of reflector i
// at row i + sb_band(), zeros above it within its block of 128) and the stage-2 reflectors
// in work (sb_work_floats() floats).  The update problems come from sb_tables()
// (sb_table_entries() entries).  Matrices m0 .. m1-1 of the batch.
struct SbArgs {
  float *A;
  int64_t mat_stride;
  int32_t n;
  int32_t spin_max;      // bound of one dependency wait of the bulge chase (0: the first wait
                         // gives up); a chase that gives up leaves NaN on the diagonal
  float *work;
  int64_t work_stride;
  double *d, *e;
  float *tau;
};
constexpr int SB_MAX_N = 8192;
constexpr int SB_SPIN_DEFAULT = 1 << 24;
int sb_band();
size_t sb_work_floats(int n_mat, int n);
size_t sb_table_entries(int n_mat, int n);
void sb_tables(const EigBatch &b, float *work, GemmProblem *tab_host);
hipError_t launch_sb_reduce(const EigBatch &b, float *work, const GemmProblem *tab_dev, hipStream_t st,
                            int m0 = 0, int m1 = -1, int spin_max = SB_SPIN_DEFAULT);
// U (fp32, first k[mat] columns) = Q2 Z for the tridiagonal's eigenvectors Z of w.
hipError_t launch_sb_q2(const EigBatch &b, const float *work, const InvitWork &w, int kmax, float *U, int64_t ldu,
                        int64_t u_stride, hipStream_t st);

// ----------------------------------------------------------------- serialisation
struct SerCell {
  const float *G;          // core, slice s at G + s * g_slice_stride, row r at + r * g_ld
  int64_t g_slice_stride, g_ld;
  void *G_out;             // blob core section (m x r_T x r_d, fp16 or fp32)
  int8_t *gexp;            // blob exponent section (m)
  int32_t r_T, r_d, f16, pad;
};
struct SerCore {
  const SerCell *cells;
  int32_t m;
};
hipError_t launch_core_pack(const SerCore &a, int n_cells, hipStream_t st);

struct SerFactorCell {
  const float *src;
  int64_t ld;
  void *dst;
  int32_t rows, cols, f16, pad;
};
struct SerFactor {
  const SerFactorCell *cells;
};
hipError_t launch_factor_pack(const SerFactor &a, int n_cells, int64_t max_elems, hipStream_t st);

// ----------------------------------------------------------------- FlashJoLT
struct SketchArgs {
  const uint64_t *seeds;    // device [n_cells]
  uint16_t *out;            // bf16 bits, [cell][N][ld]
  int64_t cell_stride;
  int32_t N, l, ld, pad;
};
hipError_t launch_sketch(const SketchArgs &a, int n_cells, hipStream_t st);

struct Gram64Args {
  const float *Y;           // [cell] rows x ld (first l columns used)
  int64_t y_cell_stride, ld;
  int32_t rows, l, chunks, chunk_rows;
  double *partial;          // [cell][chunks][l][l]
  double *G;                // [cell][l][l] (lower triangle written)
};
int gram64_tile();
hipError_t launch_gram64(const Gram64Args &a, int n_cells, hipStream_t st);
// G[cell] = (double) C[cell], both [cell][l][l]
hipError_t launch_widen_gram(const float *C, double *G, int l, int n_cells, hipStream_t st);
// sum of n_split partial lower-triangle Grams per cell into the full symmetric fp64 Gram
hipError_t launch_sum_gram_parts(const float *part, double *G, int l, int n_split, int n_cells, hipStream_t st);

struct CholArgs {
  double *G;                // [cell][l][l] in: Gram (lower); out: Cholesky factor L (lower)
  double *M;                // [cell][l][l] out: L^-1 (lower)
  float *Rinv;              // [cell][l][ldr] out: L^-T (upper triangular), zero padding
  double *Dinv;             // [cell][nbk][64][64] scratch: inverses of the diagonal tiles
  double *dmax;             // [cell] scratch: largest diagonal entry of G
  int32_t *clamped;         // [cell] out: pivots raised to the floor in this factorisation
  int32_t l, ldr, nbk, pad; // nbk = chol_blocks(l)
};
int chol_blocks(int l);
hipError_t launch_chol_inv(const CholArgs &a, int n_cells, hipStream_t st);
