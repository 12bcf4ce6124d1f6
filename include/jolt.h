/*
 * jolt.h - C ABI of the MI355X (gfx950) implementation of the JoLT / FlashJoLT
 * KV-cache compression path ("A JoLT for the KV Cache", arXiv 2607.12550).
 *
 * What is computed (one "cell" = one layer group's keys or values, section 4):
 *   X in R^{m x T x d}, m = layers_in_group * heads, slice s = layer * n_heads + head.
 *   jolt_spectrum   : energy E = ||X||_F^2, token-mode spectrum (exact Gram
 *                     eigenvalues, section 4 "Partial Tucker backbone", or the
 *                     FlashJoLT randomized SVD with tail-mass accounting,
 *                     section 5) and feature-mode spectrum.
 *   jolt_allocate   : eq. (1)-(4): byte model, error model, Lagrangian
 *                     bisection choosing (r_T, r_d, b) per cell under a budget.
 *   jolt_compress   : ST-HOSVD truncation at (r_T, r_d), fp16 factor
 *                     serialisation (section 9), residual R = X - X~ against the
 *                     stored factors, randomized Hadamard rotation and b-bit
 *                     group quantisation (section 4 "Rotated residual").
 *   jolt_decompress : X^ = X~ + rotation^-1(dequantised residual).
 *
 * Conventions shared by every entry point:
 *   - Return JOLT_OK (0) or a negative JOLT_E_* code; jolt_last_error() gives a
 *     thread-local message for the last failure.  No C++ exception crosses the ABI.
 *   - Every argument is validated on the host before any device work is queued.
 *   - Device memory is owned by the caller: input tensors, blobs, outputs and the
 *     workspace.  The library never allocates device memory.
 *   - Device work is queued on the caller's stream (a hipStream_t passed as
 *     jolt_stream; NULL = the default stream).  jolt_spectrum synchronises that
 *     stream because it returns host arrays; the other calls are asynchronous.
 *   - A call processes n_cells cells of one shape (one jolt_cell_desc) together:
 *     their kernels are batched, so per-cell host arrays have n_cells entries.
 *   - Pointer arrays (X, blobs, Xhat) are host arrays of device pointers.
 */
#ifndef JOLT_H
#define JOLT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct jolt_ctx jolt_ctx;
typedef void *jolt_stream; /* hipStream_t */

enum {
  JOLT_OK = 0,
  JOLT_E_INVAL = -1,       /* bad argument (null pointer, out-of-range value) */
  JOLT_E_UNSUPPORTED = -2, /* valid but not supported (d outside {32, 64, 128}, exact
                              spectrum beyond T = 8192, sketch wider than 1024, not gfx950) */
  JOLT_E_WORKSPACE = -3,   /* workspace or blob buffer too small */
  JOLT_E_BLOB = -4,        /* corrupt or mismatched blob header */
  JOLT_E_HIP = -5,         /* HIP runtime error (message has the HIP error string) */
  JOLT_E_NONFINITE = -6,   /* input contains NaN or Inf */
  JOLT_E_STATE = -7,       /* call sequence error (e.g. stale spectrum reuse) */
  JOLT_E_NOCONV = -8       /* a solver missed its accuracy check (outputs then unreliable):
                              inverse iteration left an eigenvector whose solution growth
                              |(T - lambda I)^-1 x|_inf |T| stayed below 1e4 sqrt(n) (residual
                              above 1e-4 |T|), or, in a cell of nonzero energy, the second
                              pass of a FlashJoLT CholeskyQR2 met a pivot below its floor
                              although the first pass met none (the first pass lost rank:
                              its output is orthonormal in exact arithmetic).  Clamped pivots
                              of a first pass are the designed treatment of a rank-deficient
                              sketch (the missing directions get zero Ritz values) and are not
                              an error. */
};

enum { JOLT_F32 = 0, JOLT_BF16 = 1 };            /* element types of caches and outputs */
enum { JOLT_EXACT = 0, JOLT_FLASH = 1 };         /* token-mode method */
enum { JOLT_FACTOR_F32 = 0, JOLT_FACTOR_F16 = 1 };/* stored factor precision (c = 4 / 2) */

/* Shape and memory layout of one cell; cells passed together share it.
 * Element (slice s, token t, feature f) of a cell whose base pointer is P lives at
 *   P + (s / n_heads) * stride_layer + (s % n_heads) * stride_head + t * stride_token + f
 * (strides in elements).  Features are contiguous. */
typedef struct {
  int32_t dtype;        /* JOLT_F32 or JOLT_BF16 */
  int32_t n_layers;     /* layers in the group (>= 1) */
  int32_t n_heads;      /* heads per layer (>= 1); m = n_layers * n_heads */
  int32_t T;            /* tokens (>= 1) */
  int32_t d;            /* features (head dimension): 32, 64 or 128 */
  int32_t reserved;
  int64_t stride_layer;
  int64_t stride_head;
  int64_t stride_token; /* >= d */
} jolt_cell_desc;

/* Options of the token-mode spectrum (section 5 for the FlashJoLT fields). */
typedef struct {
  int32_t method;      /* JOLT_EXACT or JOLT_FLASH */
  int32_t q;           /* FlashJoLT kept directions; 0 = cap policy jolt_q_cap(T, ratio) */
  double ratio;        /* target compression ratio R read by the cap policy */
  int32_t oversample;  /* p: sketch width l = min(q + p, T, m*d) */
  int32_t power_iters; /* power (subspace) iterations of the range finder */
  int32_t reuse;       /* jolt_compress only.  1: take the token spectrum that the last
                          jolt_spectrum or jolt_compress call on this workspace left there
                          for these same cells, options and seeds (JOLT_E_STATE if the
                          context recorded none); the caller guarantees that the workspace
                          was neither written nor freed since.  0: compute it. */
  int32_t r_max;       /* widest token factor kept (section 4 keeps the top token
                          eigenvectors up to the largest admissible r_T): 0 = min(T, m d)
                          (exact) or q (FlashJoLT); > 0 caps it, so r_T <= r_max and the
                          workspace shrinks accordingly.  The eigenvalues returned are
                          unaffected (exact: all T; FlashJoLT: q and the tail). */
} jolt_spectrum_opts;

/* Per-cell compression parameters. */
typedef struct {
  int32_t r_T, r_d;     /* Tucker ranks; r_T = 0 iff r_d = 0 (no backbone) */
  int32_t bits;         /* residual bits b in {0, 2, 4, 8}; 0 stores no residual */
  int32_t group;        /* quantiser group size g: divides d, multiple of 8 */
  int32_t factor_dtype; /* JOLT_FACTOR_F16 (c = 2) or JOLT_FACTOR_F32 (c = 4) */
  int32_t reserved;
  uint64_t seed;        /* rotation signs; for FlashJoLT also the sketch (must equal
                           the seed given to jolt_spectrum when its result is reused) */
} jolt_params;

/* Host-side description of one cell's spectra for the allocator. */
typedef struct {
  int32_t m, T, d;
  int32_t c;             /* bytes per stored factor scalar */
  int32_t g;             /* quantiser group size */
  int32_t n_lam_T;       /* entries of lam_T */
  int32_t rT_max;        /* largest admissible r_T */
  int32_t pool;          /* budget pool (e.g. 0 = keys, 1 = values) for JOLT_ALLOC_GREEDY */
  double E;              /* ||X||_F^2 */
  const double *lam_T;   /* token-mode eigenvalues, descending (FlashJoLT: q_eff values
                            followed by the synthetic tail) */
  const double *lam_d;   /* d feature-mode eigenvalues, descending */
  int32_t n_mu;          /* 0: eq. (2)'s tau is the additive mode-tail bound
                            min(1, tau_T(r_T) + tau_d(r_d)).  > 0: mu holds n_mu rows of d
                            truncated feature spectra (jolt_truncated_spectra, row k at
                            r_T = (k + 1) * step of the allocation's grid step) and tau is
                            the exact ST-HOSVD value (E - sum_{i < r_d} mu_k[i]) / E,
                            clipped to [0, 1]; the r_T grid then ends at n_mu * step */
  int32_t reserved;
  const double *mu;      /* host, n_mu x d, rows descending; NULL when n_mu = 0 */
} jolt_cell_spectrum;

typedef struct {
  double budget_bytes;
  double eps2[4];        /* eps^2(b) for b = 0, 2, 4, 8 (eps2[0] is 1) */
  int32_t bit_mask;      /* allowed b: bit 0 -> 0, bit 1 -> 2, bit 2 -> 4, bit 3 -> 8 */
  int32_t step;          /* rank grid step (ranks are multiples of step) */
  int32_t floor_rT, floor_rd, floor_bits; /* per-cell floors (0 = none) */
  int32_t count_scale_bytes;              /* 1: add 2 bytes per quantiser group to s */
  int32_t strategy;      /* JOLT_ALLOC_JOINT (0, the default) or an ablation allocator */
} jolt_alloc_opts;

/* Allocation strategies.  JOINT is the Lagrangian dual of eq. (3)-(4).  The others are
 * the simpler schemes of the section 7 ablations (A1, A5), on the same grid, costs and
 * model errors:
 *   RANK_ONLY: the joint dual without residual (only b = 0 is allowed);
 *   GREEDY:    every cell starts at its cheapest grid point and the upgrade with the
 *              largest model-error reduction per extra byte is taken repeatedly (a cell's
 *              upgrades walk its Pareto frontier one point at a time; upgrades that do not
 *              fit are skipped; equal efficiencies go to the lower cell index).  No global
 *              multiplier: each pool (jolt_cell_spectrum.pool) spends its own share of the
 *              budget, proportional to its cells' m T d;
 *   UNIFORM:   one (r_T, r_d, b) for every cell, the one of least summed model error whose
 *              summed cost fits (ties to the smaller cost, then b, r_T, r_d).
 * lambda_star is 0 for GREEDY and UNIFORM. */
enum { JOLT_ALLOC_JOINT = 0, JOLT_ALLOC_GREEDY = 1, JOLT_ALLOC_RANK_ONLY = 2, JOLT_ALLOC_UNIFORM = 3 };

const char *jolt_last_error(void);

/* Context: device properties only.  device < 0 uses the current device. */
int jolt_create(jolt_ctx **ctx, int device);
int jolt_destroy(jolt_ctx *ctx);

/* Section 5 "Cap selection": min(max(q_min(R), ceil(T / 32)), 512),
 * q_min = 32 for R <= 4 else 64.  Returns q (>= 1) or JOLT_E_INVAL. */
int jolt_q_cap(int T, double ratio);

/* Length of the lam_T array jolt_spectrum returns per cell (T for the exact
 * method, q_eff + 1 for FlashJoLT) and the largest admissible r_T. */
int jolt_spectrum_len(const jolt_cell_desc *desc, const jolt_spectrum_opts *opts,
                      int32_t *n_lam_T, int32_t *rT_max);

/* Device workspace (bytes) needed by jolt_spectrum and jolt_compress for n_cells
 * cells of this shape and method (opts NULL = exact method).  The same workspace
 * also serves jolt_decompress of the blobs those calls write.  Errors: as
 * jolt_spectrum's validation of desc/opts. */
int jolt_workspace_size(const jolt_cell_desc *desc, int n_cells, const jolt_spectrum_opts *opts,
                        size_t *bytes);

/* Device workspace (bytes) jolt_decompress needs for n_cells blobs of shape out_desc
 * whose largest token rank is max_rT (callers that only decode need no more). */
int jolt_decompress_workspace_size(const jolt_cell_desc *out_desc, int n_cells, int max_rT,
                                   size_t *bytes);

/* Token- and feature-mode spectra of every cell (section 4, "Partial Tucker
 * backbone"; section 5 for JOLT_FLASH).
 *   X[i]    device pointer to cell i, laid out by desc; read only.
 *   seeds   host array of n_cells sketch seeds (Philox key of the FlashJoLT Gaussian
 *           test matrix); required for JOLT_FLASH, ignored (may be NULL) otherwise.
 *   E       host, n_cells: ||X||_F^2 (fp64 sums).
 *   lam_T   host, n_cells x n_lam_T (jolt_spectrum_len), descending, clipped at 0:
 *           exact - all T eigenvalues of X_(2) X_(2)^T;  FlashJoLT - the q_eff Ritz
 *           values of the sketch followed by the synthetic tail E - sum(captured).
 *   lam_d   host, n_cells x d: eigenvalues of sum_s X_s^T X_s, descending.
 *   ws      device workspace of jolt_workspace_size bytes, 256-byte aligned; it keeps
 *           the token factors, so a later jolt_compress of the same cells with the same
 *           workspace, options and seeds can skip the spectrum (opts->reuse = 1).  The
 *           context records one spectrum per workspace; any call that writes an
 *           overlapping workspace (jolt_spectrum, jolt_compress, jolt_decompress,
 *           jolt_eps2_calibrate) first drops the record.
 * Synchronises the stream (the outputs are host arrays).  Errors: JOLT_E_INVAL
 * (null/misaligned pointers), JOLT_E_WORKSPACE, JOLT_E_NONFINITE (a cell holds NaN or
 * Inf; outputs then undefined), JOLT_E_NOCONV (see its definition), JOLT_E_UNSUPPORTED,
 * JOLT_E_HIP. */
int jolt_spectrum(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                  const uint64_t *seeds, const jolt_spectrum_opts *opts, void *ws, size_t ws_bytes,
                  double *E, double *lam_T, double *lam_d, jolt_stream stream);

/* Bytes of one cell's blob: eq. (1)'s payload (the factors at c bytes per scalar, with
 * c = 2 for the fp16 serialisation of section 9, and b/8 bytes per residual entry) plus
 * what the format adds to it: a 128-byte header, 256-byte alignment of every section, the
 * m int8 core exponents and the fp16 group scales (2 bytes per g entries).  Sections:
 * U_T (T x r_T), U_d (d x r_d), G (m x r_T x r_d) at c bytes per scalar (fp16 or fp32,
 * row-major), the core exponents (fp16 cores are stored as G_s / 2^e_s), the scales
 * (m*T*d/g) and the b-bit codes (m*T*d*b/8 bytes, packed LSB first).  Errors:
 * JOLT_E_INVAL / JOLT_E_UNSUPPORTED for a bad descriptor or parameters. */
int jolt_compressed_size(const jolt_cell_desc *desc, const jolt_params *params, size_t *bytes);

/* Compresses every cell into its blob (section 4): ST-HOSVD truncation to (r_T, r_d)
 * with the token mode first, factors rounded to the stored precision, residual
 * R = X - X~ against the stored factors, randomized Hadamard rotation of every
 * feature row and b-bit symmetric group quantisation.
 *   params  host, n_cells; group and factor_dtype must be equal across the call.
 *   blobs   device pointers (256-byte aligned) to blob_bytes[i] >= jolt_compressed_size
 *           bytes each; written completely (header included), owned by the caller.
 * Synchronises the stream before returning, to read the input and solver checks
 * (JOLT_E_NONFINITE when the call computed the spectrum itself and a cell holds NaN or
 * Inf; JOLT_E_NOCONV; the blobs are then undefined).  Errors: as jolt_spectrum, plus
 * JOLT_E_WORKSPACE for a short blob and JOLT_E_INVAL for ranks above jolt_spectrum_len's
 * rT_max. */
int jolt_compress(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                  const jolt_params *params, const jolt_spectrum_opts *opts, void *ws,
                  size_t ws_bytes, void *const *blobs, const size_t *blob_bytes,
                  jolt_stream stream);

/* Reconstructs every blob (section 4, decoding): X^ = U_T G_s U_d^T + rotation^-1 of the
 * dequantised residual, written to Xhat[i] (device, 16-byte aligned) laid out by
 * out_desc, whose dtype is the output type (JOLT_BF16 rounds to nearest even,
 * JOLT_F32 keeps fp32).  The blobs' shapes must equal out_desc's.  hdr_host (optional,
 * may be NULL) is a host copy of the n_cells 128-byte headers; without it the headers
 * are copied device->host, which synchronises the stream.  ws: at least
 * jolt_decompress_workspace_size bytes.  Errors: JOLT_E_BLOB for a corrupt or
 * mismatched header (checked before any device work), JOLT_E_WORKSPACE, JOLT_E_INVAL. */
int jolt_decompress(jolt_ctx *ctx, int n_cells, const void *const *blobs, const size_t *blob_bytes,
                    const void *hdr_host, const jolt_cell_desc *out_desc, void *const *Xhat,
                    void *ws, size_t ws_bytes, jolt_stream stream);

/* Rotary position embedding applied while decoding (appendix B: keys are compressed
 * before RoPE and the rotation is re-applied at decode time).  Feature pairs (j, j + d/2)
 * of token t rotate by the angle (t + position_offset) * base^(-2 j / d), j < d/2
 * (the half-split pairing of the Mistral / LLaMA checkpoints):
 *   x'_j = x_j cos - x_{j+d/2} sin,   x'_{j+d/2} = x_{j+d/2} cos + x_j sin.
 * Angles are formed and reduced in fp64; the rotation is applied in fp32 to the decoded
 * values before the output cast. */
typedef struct {
  double base;             /* e.g. 1e4 (LLaMA-2) or 1e6 (Mistral-7B-v0.3); must be > 1 */
  int32_t position_offset; /* position of token 0 of every cell (>= 0) */
  int32_t reserved;
} jolt_rope;

/* jolt_decompress with the rotary embedding above applied to every decoded row (rope
 * NULL: identical to jolt_decompress).  Errors: as jolt_decompress, plus JOLT_E_INVAL
 * for base <= 1 or a negative offset. */
int jolt_decompress_rope(jolt_ctx *ctx, int n_cells, const void *const *blobs, const size_t *blob_bytes,
                         const void *hdr_host, const jolt_cell_desc *out_desc, void *const *Xhat,
                         const jolt_rope *rope, void *ws, size_t ws_bytes, jolt_stream stream);

/* Budgeted allocation (section 4, eq. (1)-(4); host only, no device work): for every
 * cell the grid point (r_T, r_d, b) minimising eq. (2)'s model error plus lambda times
 * eq. (1)'s bytes, with lambda found by bisection so that the summed bytes meet the
 * budget (opts->strategy selects an ablation allocator instead, see JOLT_ALLOC_*).
 * Outputs (host, n_cells each) r_T, r_d, bits; lambda_star, total bytes and summed
 * model error.  *infeasible is 1 when even the cheapest grid point of every cell (of a
 * pool, for GREEDY) exceeds the budget (the cheapest allocation is then returned). */
int jolt_allocate(const jolt_cell_spectrum *cells, int n_cells, const jolt_alloc_opts *opts,
                  int32_t *r_T, int32_t *r_d, int32_t *bits, double *lambda_star,
                  double *total_bytes, double *model_error, int32_t *infeasible);

/* Eq. (2) calibration: eps^2(b) for b = 0, 2, 4, 8 from a round trip of n_samples
 * Gaussian samples (rows of d, group g, Philox seed).  n_samples must be a
 * multiple of d.  ws: at least jolt_eps2_workspace_size bytes. */
int jolt_eps2_workspace_size(int d, int n_samples, size_t *bytes);
int jolt_eps2_calibrate(jolt_ctx *ctx, int group, int d, uint64_t seed, int n_samples,
                        double eps2_out[4], void *ws, size_t ws_bytes, jolt_stream stream);

/* Truncated feature spectra: the exact ST-HOSVD truncation error of every grid point
 * (section 4, eq. (2)'s tau; the token mode is truncated first).  For every cell and
 * every r_T = step, 2 step, ..., n_r * step, the d eigenvalues (descending, clipped at 0)
 * of F_Y(r_T) = sum_s Y_s^T Y_s with Y_s = U_r^T X_s and U_r the first r_T columns of the
 * token factor (exact method: top eigenvectors of the token Gram; FlashJoLT: Q W).  With
 * orthonormal factors the truncation at (r_T, r_d) keeps exactly the top r_d of them, so
 * jolt_allocate takes tau = (E - their sum) / E from these rows (jolt_cell_spectrum.mu).
 * Y is formed once at r_T = n_r * step; F_Y(k step) is the running sum over k of the
 * Grams of its row blocks k (fp32 per block, fp64 running sums, fp32 matrices), then
 * diagonalised by the one-workgroup tridiagonalisation and fp64 bisection.
 *   X, seeds, opts, stream: as jolt_spectrum.  opts->reuse = 1 takes the token spectrum a
 *         jolt_spectrum or jolt_compress call left in this same workspace for these cells
 *         (JOLT_E_STATE if there is none); 0 computes it (and records it, as jolt_spectrum).
 *   step, n_r   step >= 1, n_r >= 1, n_r * step <= rT_max of jolt_spectrum_len.
 *   mu    host, n_cells x n_r x d doubles.
 *   ws    device, 256-byte aligned, at least jolt_truncated_spectra_workspace_size bytes,
 *         owned by the caller; its first jolt_workspace_size bytes are laid out as the
 *         spectrum workspace of the same cells, so a spectrum reused from it must have
 *         been computed with this same ws and ws_bytes.
 * Synchronises the stream.  Errors: as jolt_spectrum (JOLT_E_NONFINITE when the call
 * computed the spectrum itself), plus JOLT_E_INVAL for step or n_r out of range. */
int jolt_truncated_spectra_workspace_size(const jolt_cell_desc *desc, int n_cells,
                                          const jolt_spectrum_opts *opts, int step, int n_r,
                                          size_t *bytes);
int jolt_truncated_spectra(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                           const uint64_t *seeds, const jolt_spectrum_opts *opts, int step, int n_r,
                           void *ws, size_t ws_bytes, double *mu, jolt_stream stream);

/* Three-mode spectral diagnostics (section 3 and appendix A).  The token- and
 * feature-mode spectra of a cell are jolt_spectrum's (exact method: all T eigenvalues
 * of X_(2) X_(2)^T, all d of F); the slice mode completes the three unfoldings.
 *
 * jolt_slice_spectrum: for each cell, all m = n_layers * n_heads eigenvalues, descending
 * and clipped at 0, of the slice Gram S[s][s'] = sum_{t,f} X[s][t][f] X[s'][t][f] (the
 * squared singular values of the slice unfolding; for one layer, the head mode).  The
 * Gram is accumulated per token in fp32 and across tokens in fp64, reduced over token
 * chunks in a fixed order, and diagonalised by the one-workgroup tridiagonalisation and
 * fp64 bisection.  Cells, strides and X as for jolt_spectrum; m <= 768
 * (JOLT_E_UNSUPPORTED otherwise).  lam_s: host, n_cells x m doubles.  ws: device,
 * 256-byte aligned, at least jolt_slice_spectrum_workspace_size bytes, owned by the
 * caller.  Synchronises the stream. */
int jolt_slice_spectrum_workspace_size(const jolt_cell_desc *desc, int n_cells, size_t *bytes);
int jolt_slice_spectrum(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                        void *ws, size_t ws_bytes, double *lam_s, jolt_stream stream);

/* Appendix-A summary of one mode spectrum (host only): lam holds the n squared singular
 * values of an n-row unfolding, descending, >= 0.  sigma_range = sqrt(lam[0] / lam[n-1])
 * (+inf when lam[n-1] is 0); rank_a / rank_b = the smallest r in 0..n with
 * sqrt(sum_{i >= r} lam[i] / sum_i lam[i]) <= err_a / err_b (the relative Frobenius error
 * of keeping the top r; 0 when the spectrum is all zero).  JOLT_E_INVAL for n < 1, null
 * pointers, a negative or increasing spectrum, or a threshold outside [0, 1]. */
int jolt_mode_summary(const double *lam, int n, double err_a, double err_b, double *sigma_range,
                      int32_t *rank_a, int32_t *rank_b);

/* Decode-time attention evaluated on the compressed factors (section 8 and the
 * conclusion: attention run directly on the factors, without materialising the cache).
 * Item i pairs a key blob and a value blob of the same cell shape (as written by
 * jolt_compress, any ranks and bits) with a layer index layers[i] of that cell's group and
 * n_q query heads; with H key-value heads per layer (n_q a multiple of H), query head j
 * reads slice s = layers[i] * H + j / (n_q / H).  The result is
 *   O[i][j] = sum_t softmax_t(scale * Q[i][j] . K^[s][t]) V^[s][t],
 * with K^ and V^ the cells jolt_decompress would return in fp32, computed without forming
 * them: the key scores are U_T (2^e G_s U_d^T q) plus the dequantised codes dotted with
 * the query rotated once (H (signs . q) / sqrt(d)), and the value side sums U_T rows and
 * dequantised codes under the softmax weights before the value factors and the inverse
 * rotation are applied once per head.  fp32 arithmetic; chunks of 64 tokens are merged
 * with the max / rescale rule in a fixed order (deterministic).  Keys are used as stored
 * (no position rotation is applied).
 * k_hdr_host / v_hdr_host: host copies of the n_items 128-byte blob headers (validated
 * before any device work); blobs, Q ([n_items][n_q][d] fp32) and O (same shape) are device
 * memory owned by the caller; all items share m, T, d, H and the quantiser group; ranks at
 * most 1024, n_q at most 64, at most 8 query heads per key-value head and T at most 524288
 * (JOLT_E_UNSUPPORTED).  ws: device, 256-byte aligned, at least
 * jolt_attend_workspace_size bytes (max_rT_k / max_rT_v: largest key / value r_T of the
 * call).  Asynchronous on the stream. */
int jolt_attend_workspace_size(int n_items, int n_q, int T, int d, int max_rT_k, int max_rT_v,
                               size_t *bytes);
int jolt_attend(jolt_ctx *ctx, int n_items, const void *const *k_blobs, const size_t *k_bytes,
                const void *const *v_blobs, const size_t *v_bytes, const void *k_hdr_host,
                const void *v_hdr_host, const int32_t *layers, int n_q, const float *Q, float scale,
                float *O, void *ws, size_t ws_bytes, jolt_stream stream);

/* jolt_attend without a caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Arguments, result and errors as jolt_attend; the workspace is a fixed scratch array of
 * JOLT_ATTEND_SCRATCH_BYTES bytes that the library holds on every device it runs on until
 * the process ends (its address is resolved once per device by jolt_create).  Calls whose
 * jolt_attend_workspace_size exceeds it fail with JOLT_E_WORKSPACE before any device work
 * (split the items over several calls).  The call allocates nothing.  Every call on a
 * device shares that device's scratch and it keeps the last call's contents (each call
 * writes every part it reads), so calls that overlap on one device race: serialise them
 * (one stream, or events) across threads and contexts of the same device. */
#define JOLT_ATTEND_SCRATCH_BYTES (64u << 20)
int jolt_attend_noalloc(jolt_ctx *ctx, int n_items, const void *const *k_blobs, const size_t *k_bytes,
                        const void *const *v_blobs, const size_t *v_bytes, const void *k_hdr_host,
                        const void *v_hdr_host, const int32_t *layers, int n_q, const float *Q,
                        float scale, float *O, jolt_stream stream);

/* Test hook: copies an intermediate of the most recent jolt_compress on this
 * context for cell `cell` into dst (device memory, dst_bytes): 0 = U_T (T x r_T fp32),
 * 1 = U_d (d x r_d fp32), 2 = X~ (m x T x d fp32 from the stored factors, recomputed by
 * the call's own fused reconstruction in an export mode: the residual pass never stores
 * it; dst 16-byte aligned), 3 = FlashJoLT sketch Omega (m*d x l, bf16 bits).  Requires the
 * workspace and the blobs of that call to be untouched since. */
int jolt_debug_export(jolt_ctx *ctx, int what, int cell, void *dst, size_t dst_bytes,
                      jolt_stream stream);

/* Test and tuning hooks on a context.  JOLT_DBG_INVIT_ITERS forces a solver condition from
 * the host so that the JOLT_E_NOCONV path can be exercised with inputs on which the solvers
 * succeed: it sets the number of inverse-iteration sweeps of later calls on this context
 * (default 2, range 0..8; with 0 no sweep runs and the growth check fails).
 * JOLT_DBG_TRD_LANES sets how many streams the blocked tridiagonalisation of the exact token
 * spectrum spreads its groups of matrices over (default 4, range 1..4; results do not
 * depend on it): 1 keeps every launch on the call's stream, for counter collection.
 * JOLT_DBG_TRD_TWO_STAGE selects the reduction of those large matrices to tridiagonal form:
 * 1 the two-stage reduction (dense to a band of half-bandwidth 32 by panel QR and
 * matrix-core updates, then bulge chasing), 0 the one-stage blocked Householder reduction,
 * -1 (default) two stages when the call's matrices times their order reach 32 * 4096, one
 * otherwise; both give the same spectrum and projectors to rounding, and a compress that
 * reuses a recorded spectrum back-transforms with the reduction that made it.
 * JOLT_DBG_BULGE_SPIN bounds each dependency wait of the two-stage reduction's bulge chase
 * (default 2^24 polls, range 0..2^24; 0 makes the first wait give up): a chase that gives up
 * ends normally and the call reports JOLT_E_NOCONV, which lets that path be exercised.
 * Errors: JOLT_E_INVAL. */
enum { JOLT_DBG_INVIT_ITERS = 0, JOLT_DBG_TRD_LANES = 1, JOLT_DBG_TRD_TWO_STAGE = 2, JOLT_DBG_BULGE_SPIN = 3 };
int jolt_debug_set(jolt_ctx *ctx, int what, int64_t value);

/* Benchmark instrumentation.  When enabled, the library brackets the kernels of each
 * stage below with one pair of HIP events per stage and call, recorded on the call's
 * stream; jolt_profile_read waits for the recorded events and returns the device time (ms)
 * accumulated since the last reset and the number of bracketed intervals.  At most 4096
 * intervals are kept pending: beyond that the oldest are read (a host wait).  Disabled by
 * default (no events). */
enum {
  JOLT_STAGE_FEATURE_GRAM = 0, /* E and F = sum_s X_s^T X_s (and F_Y during ST-HOSVD) */
  JOLT_STAGE_TOKEN_GRAM,       /* C = X_(2) X_(2)^T */
  JOLT_STAGE_TRIDIAG_LARGE,    /* blocked tridiagonalisation of token Grams with T > 768 (mat-vec
                                  tiles, per-column kernels and rank-2k updates, replayed as one
                                  graph and timed as a whole) */
  JOLT_STAGE_RESERVED_3,       /* not recorded */
  JOLT_STAGE_RESERVED_4,       /* not recorded */
  JOLT_STAGE_TRIDIAG_SMALL,    /* one-workgroup tridiagonalisation (small n) */
  JOLT_STAGE_EIGVALS,          /* fp64 bisection */
  JOLT_STAGE_EIGVECS,          /* fp64 inverse iteration + cluster re-orthogonalisation */
  JOLT_STAGE_BACKTRANSFORM,    /* U = Q Z */
  JOLT_STAGE_PROJECT,          /* Y = U_T^T X_(2) */
  JOLT_STAGE_CORE,             /* G_s = Y_s U_d */
  JOLT_STAGE_SERIALIZE,        /* factor and core packing */
  JOLT_STAGE_RECONSTRUCT,      /* W_s and X~_s = U_T W_s from the stored factors */
  JOLT_STAGE_RESIDUAL,         /* residual, rotation, quantisation, packing */
  JOLT_STAGE_DECODE,           /* dequantisation, inverse rotation, add, cast */
  JOLT_STAGE_SKETCH,           /* FlashJoLT sketch products */
  JOLT_STAGE_ORTH,             /* FlashJoLT orthonormalisation */
  JOLT_STAGE_SLICE_GRAM,       /* slice-mode Gram of the three-mode diagnostics */
  JOLT_STAGE_ATTEND,           /* decode attention on the factors */
  JOLT_STAGE_TRUNC_GRAM,       /* prefix feature Grams of the token-truncated cell */
  JOLT_STAGE_COUNT
};
int jolt_profile_enable(jolt_ctx *ctx, int on);
int jolt_profile_reset(jolt_ctx *ctx);
int jolt_profile_read(jolt_ctx *ctx, int stage, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* JOLT_H */
