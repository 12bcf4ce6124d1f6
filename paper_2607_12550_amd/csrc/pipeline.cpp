// Orchestration of the compression path on the device: workspace layout, the
// spectral stage (section 4 partial Tucker spectra; section 5 FlashJoLT), the codec
// stage (ST-HOSVD truncation, fp16 serialisation, closed-loop residual, rotation,
// quantisation) and the decoder.  All cells of a call share one shape and are
// batched into the same kernel launches.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "host_util.h"
#include "jolt_internal.h"

namespace {

constexpr int KC = 512;   // inverse-iteration columns per launch (bounds its scratch)
constexpr int SYTRD_SMALL_MAX = 768;   // larger matrices use the blocked multi-workgroup kernel
constexpr int SYTRD_NB = 32;
constexpr int kG64Rows = 8192;          // rows per split-K chunk of the fp64 sketch Gram
constexpr int kGramSplitMax = 16;       // row chunks of the second CholeskyQR pass's Gram
constexpr int kOrthMax = 33;            // CholeskyQR2 calls of one spectrum (1 + 2 x 16 power iterations)

struct Carver {
  uint8_t *base;
  size_t off = 0;
  explicit Carver(void *b) : base(static_cast<uint8_t *>(b)) {}
  template <class T>
  T *take(size_t n) {
    off = (off + 255) / 256 * 256;
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

struct EigWs {
  EigBatch b{};
  double *Z = nullptr, *lu = nullptr;
  int32_t *k = nullptr;
  int32_t *status = nullptr;   // inverse-iteration convergence flags, one per matrix
  float *bt = nullptr;
  float *trd = nullptr;    // blocked tridiagonalisation work (large n only)
  int kmax = 0;
};

struct Ws {
  // tables
  GemmProblem *tab = nullptr;
  size_t tab_n = 0;
  FusedCell *fcell_r = nullptr;   // per-cell records of the fused reconstruction passes
  int32_t *wexp = nullptr;         // [cell][slice] exponents of W_s (or of U^_T G^_s)
  uint16_t *udp = nullptr;         // [cell] d x d: U^_d in the fused kernel's slot order
  FGramCell *fcell = nullptr;
  SerCell *scell = nullptr;
  SerFactorCell *sfcell = nullptr;
  uint64_t *seeds = nullptr;
  int32_t *nonfinite = nullptr;
  float *signs = nullptr;
  // feature Gram
  int chunks = 1;
  float *fpart = nullptr, *F = nullptr;
  double *epart = nullptr, *E = nullptr;
  EigWs feig;          // feature Gram of X (eigenvalues) and of Y (eigenvectors)
  float *Ud = nullptr;
  // token
  float *C = nullptr;  // exact: token Gram, flash: B B^T
  EigWs teig;
  float *U = nullptr;  // token factor, T x kmaxT per cell
  int kmaxT = 0;
  // ST-HOSVD / reconstruction
  float *Y = nullptr, *G = nullptr, *W = nullptr;   // W: W_s^T (d x ldw) per slice
  int ldw = 0;
  // FlashJoLT
  int ldo = 0, ldl = 0, g64_chunks = 0;
  uint16_t *Om = nullptr;                 // sketch, N x ldo bf16 per cell
  float *Ysk = nullptr, *Qsk = nullptr;   // T x ldl: range basis and CholeskyQR scratch
  float *Zsk = nullptr, *Qz = nullptr;    // N x ldl: power-iteration basis and scratch
  float *Bsk = nullptr;                   // l x N: B = Q^T X_(2)
  float *Wsk = nullptr;                   // l x q: Ritz vectors of B B^T
  double *g64p = nullptr, *g64 = nullptr, *chM = nullptr, *chD = nullptr, *chMax = nullptr;
  int32_t *orth_clamp = nullptr;          // [orth call][pass][cell] clamped Cholesky pivots
  float *Rinv = nullptr;                  // l x ldl
  // eps2
  double *eps_part = nullptr;
};

size_t eig_bt_floats(int nmat, int n, int kmax) { return backtransform_scratch_floats(nmat, n, kmax); }

void carve_eig(Carver &cv, EigWs &e, int nmat, int n, int kmax, float *A) {
  e.b.A = A;
  e.b.mat_stride = (int64_t)n * n;
  e.b.n_mat = nmat;
  e.b.n = n;
  e.b.d = cv.take<double>((size_t)nmat * n);
  e.b.e = cv.take<double>((size_t)nmat * n);
  e.b.lam = cv.take<double>((size_t)nmat * n);
  e.b.tau = cv.take<float>((size_t)nmat * n);
  e.kmax = kmax;
  e.k = cv.take<int32_t>(nmat);
  e.status = cv.take<int32_t>(nmat);
  if (n > SYTRD_SMALL_MAX)
    e.trd = cv.take<float>(std::max(sytrd_large_work_floats(nmat, n, SYTRD_NB), sb_work_floats(nmat, n)));
  if (kmax > 0) {
    e.Z = cv.take<double>((size_t)nmat * n * kmax);
    e.lu = cv.take<double>((size_t)nmat * 3 * n * std::min(kmax, KC));
    e.bt = cv.take<float>(eig_bt_floats(nmat, n, kmax));
  }
}

void plan(Carver &cv, Ws &w, const SpecShape &sh, int nc) {
  const int m = sh.m, T = sh.T, d = sh.d, N = sh.N;
  const int nmax = std::max({T, d, sh.ell});
  w.tab_n = 8192 + backtransform_table_entries(nc, nmax) + 4 * (size_t)nc * m +
            sytrd_large_table_entries(nc, nmax, SYTRD_NB);
  // sketch, power and CholeskyQR2 products (up to 33 orthonormalisations, each with a
  // split-K Gram of up to kGramSplitMax chunks per cell)
  if (sh.method == JOLT_FLASH) w.tab_n += (size_t)nc * (160 + 33 * kGramSplitMax);
  w.tab = cv.take<GemmProblem>(w.tab_n);
  w.fcell_r = cv.take<FusedCell>(nc);
  w.wexp = cv.take<int32_t>((size_t)nc * m);
  w.fcell = cv.take<FGramCell>(nc);
  w.scell = cv.take<SerCell>(nc);
  w.sfcell = cv.take<SerFactorCell>(2 * nc);
  w.seeds = cv.take<uint64_t>(nc);
  w.nonfinite = cv.take<int32_t>(nc);
  w.signs = cv.take<float>((size_t)nc * d);
  w.chunks = (int)std::min<int64_t>(64, std::max<int64_t>(1, (int64_t)m * T / 2048));
  w.fpart = cv.take<float>((size_t)nc * w.chunks * d * d);
  w.epart = cv.take<double>((size_t)nc * w.chunks);
  w.F = cv.take<float>((size_t)nc * d * d);
  w.E = cv.take<double>(nc);
  carve_eig(cv, w.feig, nc, d, d, w.F);
  w.Ud = cv.take<float>((size_t)nc * d * d);
  w.kmaxT = sh.rT_max;
  if (sh.method == JOLT_EXACT) {
    w.C = cv.take<float>((size_t)nc * T * T);
    carve_eig(cv, w.teig, nc, T, w.kmaxT, w.C);
  } else {
    const int l = sh.ell;
    w.ldo = (l + 7) / 8 * 8;
    w.ldl = (l + 7) / 8 * 8;
    w.C = cv.take<float>((size_t)nc * l * l);
    carve_eig(cv, w.teig, nc, l, sh.q, w.C);
    w.Om = cv.take<uint16_t>((size_t)nc * N * w.ldo);
    w.Ysk = cv.take<float>((size_t)nc * T * w.ldl);
    w.Qsk = cv.take<float>((size_t)nc * T * w.ldl);
    w.Zsk = cv.take<float>((size_t)nc * N * w.ldl);
    w.Qz = cv.take<float>((size_t)nc * N * w.ldl);
    w.Bsk = cv.take<float>((size_t)nc * l * N);
    w.Wsk = cv.take<float>((size_t)nc * l * std::max(sh.q, 1));
    w.g64_chunks = (std::max(T, N) + kG64Rows - 1) / kG64Rows;
    w.g64p = cv.take<double>((size_t)nc * w.g64_chunks * l * l);
    w.g64 = cv.take<double>((size_t)nc * l * l);
    w.chM = cv.take<double>((size_t)nc * l * l);
    w.chD = cv.take<double>((size_t)nc * chol_blocks(l) * 64 * 64);
    w.chMax = cv.take<double>(nc);
    w.orth_clamp = cv.take<int32_t>((size_t)kOrthMax * 2 * nc);
    w.Rinv = cv.take<float>((size_t)nc * l * w.ldl);
  }
  w.U = cv.take<float>((size_t)nc * T * std::max(w.kmaxT, 1));
  w.Y = cv.take<float>((size_t)nc * std::max(w.kmaxT, 1) * N);
  w.G = cv.take<float>((size_t)nc * m * std::max(w.kmaxT, 1) * d);
  w.ldw = (std::max(w.kmaxT, 1) + 7) / 8 * 8;
  w.W = cv.take<float>((size_t)nc * m * d * w.ldw);
  w.udp = cv.take<uint16_t>((size_t)nc * d * d);
}

// decode-only areas: problem table, per-cell records, rotation signs, W_s^T = 2^e U_d G_s^T
// and its exponents (X~ itself is never stored)
void plan_decode(Carver &cv, Ws &w, int m, int T, int d, int nc, int kmax) {
  (void)T;
  w.tab_n = 64 + 2 * (size_t)nc * m;
  w.tab = cv.take<GemmProblem>(w.tab_n);
  w.fcell_r = cv.take<FusedCell>(nc);
  w.wexp = cv.take<int32_t>((size_t)nc * m);
  w.seeds = cv.take<uint64_t>(nc);
  w.signs = cv.take<float>((size_t)nc * d);
  w.kmaxT = std::max(kmax, 1);
  w.ldw = (w.kmaxT + 7) / 8 * 8;
  w.W = cv.take<float>((size_t)nc * m * d * w.ldw);
  w.udp = cv.take<uint16_t>((size_t)nc * d * d);
}

int dtype_gt(int dt) { return dt == JOLT_BF16 ? GT_BF16 : GT_F32; }

GemmOperand cell_operand(const void *x, const jolt_cell_desc *d) {
  return seg_operand(x, d->stride_token, d->stride_layer, d->stride_head, d->d, d->n_heads);
}

GemmOperand plain(const void *p, int64_t ld) {
  GemmOperand o{};
  o.ptr = p;
  o.ld = ld;
  o.seg_heads = 1;
  return o;
}

struct Run {
  jolt_ctx *ctx;
  hipStream_t st;
  Ws w;
  size_t tab_used = 0;
  int orth_calls = 0;      // CholeskyQR2 calls queued by this call (their clamp counts)

  // upload a problem table into the next slice of the device table area, then launch.
  // mode 0: bf16 x bf16 on the bf16 matrix cores; mode 2: the same kernel with fp32
  // operands split into bf16 hi + lo; mode 1: fp32 MFMA.  A table the bf16 kernel's layout
  // conditions reject runs on the fp32 kernel.
  int gemm(const std::vector<GemmProblem> &probs_in, int mode, int ta, int tb, bool ak, bool bk) {
    if (probs_in.empty()) return JOLT_OK;
    if (tab_used + probs_in.size() > w.tab_n)
      return jolt_fail(JOLT_E_WORKSPACE, "GEMM problem table overflow");
    std::vector<GemmProblem> probs(probs_in);
    int bm = 128;
    bool fast = false;
    if (mode == 0 || mode == 2) {
      fast = gemm16_prepare(probs.data(), (int)probs.size(), ta, tb, ak, bk, bm);
      if (!fast) probs = probs_in;
    }
    GemmProblem *dst = w.tab + tab_used;
    tab_used += probs.size();
    HIP_OK(hipMemcpyAsync(dst, probs.data(), probs.size() * sizeof(GemmProblem),
                          hipMemcpyHostToDevice, st));
    int maxM = 0, maxN = 0;
    bool lower = false;
    for (auto &p : probs) { maxM = std::max(maxM, p.M); maxN = std::max(maxN, p.N); lower = lower || p.lower_only; }
    if (fast) HIP_OK(launch_gemm16(dst, (int)probs.size(), maxM, maxN, ta, tb, ak, bk, bm, lower, st));
    else HIP_OK(launch_gemm(dst, (int)probs.size(), maxM, maxN, 1, ta, tb, ak, bk, st));
    return JOLT_OK;
  }

  GemmProblem *tab_slice(size_t n) {
    if (tab_used + n > w.tab_n) return nullptr;
    GemmProblem *p = w.tab + tab_used;
    tab_used += n;
    return p;
  }
};

// symmetric eigenvalues (all) of the n x n matrices in e.b.A
int eig_values(Run &R, EigWs &e) {
  if (e.b.n > SYTRD_SMALL_MAX) {
    jolt_ctx *c = R.ctx;
    // Two stages (band of half-bandwidth sb_band(), then bulge chasing) move the trailing
    // matrix once per panel instead of once per column, but their bulge chase is a chain of
    // about n^2 / 64 dependent steps per matrix; the one-stage reduction costs about n^3 / 6
    // floats of trailing-matrix reads per matrix.  With the batch's matrices run side by side
    // the chain is hidden once the batch holds n_mat * n >= 32 * 4096 (measured crossover at
    // n = 4096: 16 matrices favour one stage, 64 two).  The eigenvector back-transform
    // follows the choice.
    const bool two = c->trd_two_stage == 1 ||
                     (c->trd_two_stage < 0 && (int64_t)e.b.n_mat * e.b.n >= kTwoStageMinWork);
    e.b.refl_off = two ? sb_band() : 1;
    const size_t nt = two ? sb_table_entries(e.b.n_mat, e.b.n) : sytrd_large_table_entries(e.b.n_mat, e.b.n, SYTRD_NB);
    GemmProblem *tab = R.tab_slice(nt);
    if (!tab) return jolt_fail(JOLT_E_WORKSPACE, "GEMM problem table overflow");
    c->tab_host.resize(std::max(c->tab_host.size(), nt));
    if (two) sb_tables(e.b, e.trd, c->tab_host.data());
    else sytrd_large_tables(e.b, e.trd, SYTRD_NB, c->tab_host.data());
    HIP_OK(hipMemcpyAsync(tab, c->tab_host.data(), nt * sizeof(GemmProblem), hipMemcpyHostToDevice, R.st));
    {
      // the launch sequence depends only on the shape and the buffers: capture it once per
      // group of matrices, and replay the groups side by side, the first on the caller's
      // stream and the others on private streams between a fork from and a join into it
      // (timed as one stage when profiling is on; its kernels are told apart by a kernel trace)
      std::vector<const void *> key{e.b.A, e.trd, tab, e.b.d, e.b.e, e.b.tau,
                                    reinterpret_cast<const void *>((intptr_t)e.b.n),
                                    reinterpret_cast<const void *>((intptr_t)e.b.n_mat),
                                    reinterpret_cast<const void *>((intptr_t)(two ? 2 : 1)),
                                    reinterpret_cast<const void *>((intptr_t)c->bulge_spin)};
      const int lanes = std::min(c->trd_lanes_max, e.b.n_mat);
      if (c->trd_lanes != lanes || c->trd_key != key) {
        for (int g = 0; g < jolt_ctx::kTrdLanes; ++g)
          if (c->trd_exec[g]) { HIP_OK(hipGraphExecDestroy(c->trd_exec[g])); c->trd_exec[g] = nullptr; }
        c->trd_lanes = 0;
        if (!c->trd_fork) HIP_OK(hipEventCreateWithFlags(&c->trd_fork, hipEventDisableTiming));
        for (int g = 0; g < lanes; ++g) {
          // lane 0 replays on the caller's stream and is captured on lane 1's stream (no
          // stream of its own, so that lanes + 1 streams never exceed the hardware queues)
          const int cs = g > 0 ? g : 1;
          if (!c->cap_stream[cs]) HIP_OK(hipStreamCreateWithFlags(&c->cap_stream[cs], hipStreamNonBlocking));
          if (!c->trd_join[g]) HIP_OK(hipEventCreateWithFlags(&c->trd_join[g], hipEventDisableTiming));
          const int m0 = (int)((int64_t)e.b.n_mat * g / lanes), m1 = (int)((int64_t)e.b.n_mat * (g + 1) / lanes);
          hipGraph_t gr = nullptr;
          HIP_OK(hipStreamBeginCapture(c->cap_stream[cs], hipStreamCaptureModeThreadLocal));
          hipError_t le = two ? launch_sb_reduce(e.b, e.trd, tab, c->cap_stream[cs], m0, m1, c->bulge_spin)
                              : launch_sytrd_large(e.b, e.trd, SYTRD_NB, tab, c->cap_stream[cs], m0, m1);
          hipError_t ce = hipStreamEndCapture(c->cap_stream[cs], &gr);
          HIP_OK(le);
          HIP_OK(ce);
          hipError_t ie = hipGraphInstantiate(&c->trd_exec[g], gr, nullptr, nullptr, 0);
          (void)hipGraphDestroy(gr);
          HIP_OK(ie);
        }
        c->trd_lanes = lanes;
        c->trd_key = key;
      }
      StageTimer t(R.ctx, R.st, JOLT_STAGE_TRIDIAG_LARGE);
      HIP_OK(hipEventRecord(c->trd_fork, R.st));
      for (int g = 1; g < lanes; ++g) {
        HIP_OK(hipStreamWaitEvent(c->cap_stream[g], c->trd_fork, 0));
        HIP_OK(hipGraphLaunch(c->trd_exec[g], c->cap_stream[g]));
        HIP_OK(hipEventRecord(c->trd_join[g], c->cap_stream[g]));
      }
      HIP_OK(hipGraphLaunch(c->trd_exec[0], R.st));
      for (int g = 1; g < lanes; ++g) HIP_OK(hipStreamWaitEvent(R.st, c->trd_join[g], 0));
    }
  } else {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_TRIDIAG_SMALL);
    HIP_OK(launch_sytrd_small(e.b, R.st));
  }
  StageTimer t(R.ctx, R.st, JOLT_STAGE_EIGVALS);
  HIP_OK(launch_tridiag_eigvals(e.b, R.st));
  return JOLT_OK;
}

// top-k[mat] eigenvectors into U (fp32, n x ldu per matrix at u_stride); requires eig_values first
int eig_vectors(Run &R, EigWs &e, const std::vector<int> &k, float *U, int64_t ldu, int64_t u_stride) {
  int kmax = 0;
  for (int v : k) kmax = std::max(kmax, v);
  if (kmax == 0) return JOLT_OK;
  if (kmax > e.kmax) return jolt_fail(JOLT_E_WORKSPACE, "eigenvector count %d exceeds workspace %d", kmax, e.kmax);
  HIP_OK(hipMemcpyAsync(e.k, k.data(), k.size() * sizeof(int32_t), hipMemcpyHostToDevice, R.st));
  HIP_OK(hipMemsetAsync(e.status, 0, (size_t)e.b.n_mat * sizeof(int32_t), R.st));
  InvitWork iw{e.Z, e.lu, kmax, std::min(kmax, KC), e.k, e.status, R.ctx->invit_iters, 0};
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_EIGVECS);
    HIP_OK(launch_tridiag_eigvecs(e.b, iw, kmax, R.st));
  }
  StageTimer t(R.ctx, R.st, JOLT_STAGE_BACKTRANSFORM);
  const size_t nt = backtransform_table_entries(e.b.n_mat, e.b.n);
  GemmProblem *tab = R.tab_slice(nt);
  if (!tab) return jolt_fail(JOLT_E_WORKSPACE, "GEMM problem table overflow");
  R.ctx->tab_host.resize(std::max(R.ctx->tab_host.size(), nt));
  // two-stage reduction: the band-to-tridiagonal reflectors first (Z -> U), then the
  // panel reflectors of the first stage by the blocked back-transform
  const bool two = e.b.n > SYTRD_SMALL_MAX && e.b.refl_off == sb_band();
  if (two) HIP_OK(launch_sb_q2(e.b, e.trd, iw, kmax, U, ldu, u_stride, R.st));
  HIP_OK(launch_backtransform(e.b, iw, kmax, k.data(), U, ldu, u_stride, e.bt, tab, R.ctx->tab_host.data(), R.st,
                              two));
  return JOLT_OK;
}

// Host copies of the device-side checks of one call: non-finite input cells, the clamp
// counts of every CholeskyQR2 pass and the inverse-iteration convergence flags.  queue()
// adds the copies to the stream; verdict() reads them once the stream is synchronised.
struct CallChecks {
  int nc = 0, n_orth = 0;
  bool spectrum = false;
  std::vector<int32_t> bad, clamp, tstat, fstat;
  std::vector<double> E, d0;   // d0: first diagonal entry of each two-stage tridiagonal

  int queue(Run &R, int nc_, bool spectrum_computed, bool token_vecs, bool feature_vecs) {
    nc = nc_;
    spectrum = spectrum_computed;
    if (spectrum) {
      bad.resize(nc);
      E.resize(nc);
      HIP_OK(hipMemcpyAsync(bad.data(), R.w.nonfinite, nc * sizeof(int32_t), hipMemcpyDeviceToHost, R.st));
      HIP_OK(hipMemcpyAsync(E.data(), R.w.E, nc * sizeof(double), hipMemcpyDeviceToHost, R.st));
      n_orth = R.orth_calls;
      // a bulge chase that gave up leaves NaN on its diagonal
      const EigBatch &tb = R.w.teig.b;
      if (tb.d && tb.n > SYTRD_SMALL_MAX && tb.refl_off == sb_band()) {
        d0.resize(tb.n_mat);
        HIP_OK(hipMemcpy2DAsync(d0.data(), sizeof(double), tb.d, (size_t)tb.n * sizeof(double), sizeof(double),
                                tb.n_mat, hipMemcpyDeviceToHost, R.st));
      }
      if (n_orth) {
        clamp.resize((size_t)n_orth * 2 * nc);
        HIP_OK(hipMemcpyAsync(clamp.data(), R.w.orth_clamp, clamp.size() * sizeof(int32_t),
                              hipMemcpyDeviceToHost, R.st));
      }
    }
    if (token_vecs) {
      tstat.resize(R.w.teig.b.n_mat);
      HIP_OK(hipMemcpyAsync(tstat.data(), R.w.teig.status, tstat.size() * sizeof(int32_t),
                            hipMemcpyDeviceToHost, R.st));
    }
    if (feature_vecs) {
      fstat.resize(R.w.feig.b.n_mat);
      HIP_OK(hipMemcpyAsync(fstat.data(), R.w.feig.status, fstat.size() * sizeof(int32_t),
                            hipMemcpyDeviceToHost, R.st));
    }
    return JOLT_OK;
  }

  int verdict() const {
    for (int c = 0; c < (int)bad.size(); ++c)
      if (bad[c]) return jolt_fail(JOLT_E_NONFINITE, "cell %d contains NaN or Inf", c);
    for (int c = 0; c < (int)E.size(); ++c) {
      if (!(E[c] > 0.0)) continue;
      for (int o = 0; o < n_orth; ++o) {
        const int32_t first = clamp[((size_t)o * 2 + 0) * nc + c], second = clamp[((size_t)o * 2 + 1) * nc + c];
        if (second > 0 && first == 0)
          return jolt_fail(JOLT_E_NOCONV, "cell %d: orthonormalisation %d lost rank in its first CholeskyQR "
                                          "pass (%d pivots clamped in the second)", c, o, second);
      }
    }
    for (int c = 0; c < (int)d0.size(); ++c)
      if (!std::isfinite(d0[c]))
        return jolt_fail(JOLT_E_NOCONV, "cell %d: the band-to-tridiagonal reduction of the token Gram did not complete", c);
    for (int c = 0; c < (int)tstat.size(); ++c)
      if (tstat[c]) return jolt_fail(JOLT_E_NOCONV, "cell %d: token-mode inverse iteration did not converge", c);
    for (int c = 0; c < (int)fstat.size(); ++c)
      if (fstat[c]) return jolt_fail(JOLT_E_NOCONV, "cell %d: feature-mode inverse iteration did not converge", c);
    return JOLT_OK;
  }
};

int upload_seeds_and_signs(Run &R, const uint64_t *seeds, int nc, int d) {
  HIP_OK(hipMemcpyAsync(R.w.seeds, seeds, nc * sizeof(uint64_t), hipMemcpyHostToDevice, R.st));
  HIP_OK(launch_rotation_signs(R.w.seeds, nc, d, R.w.signs, R.st));
  return JOLT_OK;
}

// E, feature Gram F (and its eigenvalues) of every cell
int feature_stage(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc,
                  const void *const *X) {
  std::vector<FGramCell> fc(nc);
  for (int c = 0; c < nc; ++c) fc[c] = FGramCell{X[c], sh.T, 0};
  HIP_OK(hipMemcpyAsync(R.w.fcell, fc.data(), nc * sizeof(FGramCell), hipMemcpyHostToDevice, R.st));
  HIP_OK(hipMemsetAsync(R.w.nonfinite, 0, nc * sizeof(int32_t), R.st));
  FGramArgs a{};
  a.cells = R.w.fcell;
  a.n_cells = nc;
  a.nseg = sh.m;
  a.seg_heads = desc->n_heads;
  a.seg_hi = desc->stride_layer;
  a.seg_lo = desc->stride_head;
  a.row_stride = desc->stride_token;
  a.chunks_per_cell = R.w.chunks;
  a.partial_F = R.w.fpart;
  a.partial_E = R.w.epart;
  a.nonfinite = R.w.nonfinite;
  // 16-byte row loads: 8-element aligned strides and 16-byte aligned cell bases
  a.vec16 = desc->stride_layer % 8 == 0 && desc->stride_head % 8 == 0 && desc->stride_token % 8 == 0;
  for (int c = 0; c < nc; ++c) a.vec16 = a.vec16 && (reinterpret_cast<uintptr_t>(X[c]) % 16 == 0);
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_FEATURE_GRAM);
    HIP_OK(launch_feature_gram(a, sh.d, desc->dtype, R.st));
    HIP_OK(launch_feature_gram_reduce(a, sh.d, R.w.F, R.w.E, R.st));
  }
  return eig_values(R, R.w.feig);
}

// exact token-mode spectrum: C = X_(2) X_(2)^T, tridiagonalise, all eigenvalues
int token_exact(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc, const void *const *X) {
  std::vector<GemmProblem> P(nc);
  for (int c = 0; c < nc; ++c) {
    GemmProblem &p = P[c];
    p = GemmProblem{};
    p.A = cell_operand(X[c], desc);
    p.B = cell_operand(X[c], desc);
    p.C = R.w.C + (size_t)c * sh.T * sh.T;
    p.ldc = sh.T;
    p.M = sh.T; p.N = sh.T; p.K = sh.N;
    p.alpha = 1.f; p.beta = 0.f;
    // the blocked tridiagonalisation reads the lower triangle (it restores the upper part of
    // each panel's rows itself), so only the lower tiles of the symmetric Gram are formed
    p.lower_only = sh.T > SYTRD_SMALL_MAX ? 1 : 0;
  }
  const int mode = desc->dtype == JOLT_BF16 ? 0 : 1;
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_TOKEN_GRAM);
    int rc = R.gemm(P, mode, dtype_gt(desc->dtype), dtype_gt(desc->dtype), true, true);
    if (rc) return rc;
  }
  return eig_values(R, R.w.teig);
}

int spectrum_device(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc,
                    const void *const *X, const uint64_t *seeds, const jolt_spectrum_opts *o);

// Sections of one blob that the reconstruction reads.
struct BlobView {
  const uint8_t *b;
  BlobLayout L;
  int rT, rd, bits;
};

// What the fused passes read besides the blobs, from the stored factors of every cell with
// a backbone.  fp16 factors: G^_s^T per slice, the exponents ky_s and the permuted U^_d
// (launch_core_prepare).  fp32 factors: W_s^T = 2^e_s U^_d G^_s^T (d x r_T per slice,
// leading dimension ldw), then the per-slice exponents k_s.
// fc: the host records of the call (uploaded here); fb: bytes per stored factor scalar.
int build_w(Run &R, int nc, int m, int d, const std::vector<BlobView> &bv, const std::vector<FusedCell> &fc,
            int fb) {
  const int ft = fb == 2 ? GT_F16 : GT_F32;
  HIP_OK(hipMemcpyAsync(R.w.fcell_r, fc.data(), nc * sizeof(FusedCell), hipMemcpyHostToDevice, R.st));
  if (fb == 2) {
    HIP_OK(launch_core_prepare(R.w.fcell_r, R.w.signs, nc, m, d, R.st));
    return JOLT_OK;
  }
  std::vector<GemmProblem> P;
  for (int c = 0; c < nc; ++c) {
    const BlobView &v = bv[c];
    if (!v.rT) continue;
    for (int s = 0; s < m; ++s) {
      GemmProblem p{};
      p.A = plain(v.b + v.L.Ud, v.rd);                                     // A(f, j) = Ud[f][j]
      p.B = plain(v.b + v.L.G + (int64_t)s * v.rT * v.rd * fb, v.rd);      // B(j, i) = G_s[i][j]
      p.C = const_cast<float *>(fc[c].Wt) + (int64_t)s * d * R.w.ldw; p.ldc = R.w.ldw;
      p.M = d; p.N = v.rT; p.K = v.rd; p.alpha = 1.f;
      p.alpha_exp2 = reinterpret_cast<const int8_t *>(v.b + v.L.gexp + s);
      P.push_back(p);
    }
  }
  int rc = R.gemm(P, 1, ft, ft, true, true);
  if (rc) return rc;
  HIP_OK(launch_w_prepare(R.w.fcell_r, nc, m, d, R.st));
  return JOLT_OK;
}

FusedCell fused_cell(Run &R, int c, int m, int d, const BlobView &v) {
  FusedCell f{};
  f.UT = v.b + v.L.UT;
  f.Wt = R.w.W + (int64_t)c * m * d * R.w.ldw;
  f.wexp = R.w.wexp + (int64_t)c * m;
  f.codes = const_cast<uint8_t *>(v.b + v.L.codes);
  f.scales = reinterpret_cast<uint16_t *>(const_cast<uint8_t *>(v.b + v.L.scales));
  f.G = reinterpret_cast<const uint16_t *>(v.b + v.L.G);
  f.gexp = reinterpret_cast<const int8_t *>(v.b + v.L.gexp);
  f.Ud = reinterpret_cast<const uint16_t *>(v.b + v.L.Ud);
  f.udp = R.w.udp + (int64_t)c * d * d;
  f.rT = v.rT; f.bits = v.bits; f.ldw = R.w.ldw; f.rd = v.rd;
  return f;
}

FusedArgs fused_args(Run &R, int nc, int m, int T, int d, int group, const jolt_cell_desc *strides) {
  FusedArgs a{};
  a.cells = R.w.fcell_r; a.signs = R.w.signs;
  a.n_cells = nc; a.m = m; a.T = T; a.heads = strides->n_heads; a.group = group;
  a.s_layer = strides->stride_layer; a.s_head = strides->stride_head; a.s_tok = strides->stride_token;
  a.inv_sqrt_d = (float)(1.0 / std::sqrt((double)d));
  return a;
}

}  // namespace

// ------------------------------------------------------------------------ sizes
void forget_spectra(jolt_ctx *ctx, const void *ws, size_t bytes, const SpecKey *keep) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(ws), a1 = a0 + bytes;
  std::vector<SpecKey> kept;
  for (SpecKey &k : ctx->specs) {
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(k.ws), b1 = b0 + k.ws_bytes;
    if (&k == keep || b1 <= a0 || a1 <= b0) kept.push_back(std::move(k));
  }
  ctx->specs.swap(kept);
}

extern "C" int jolt_workspace_size(const jolt_cell_desc *desc, int n_cells,
                                   const jolt_spectrum_opts *opts, size_t *bytes) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  if (n_cells < 1 || !bytes) return jolt_fail(JOLT_E_INVAL, "jolt_workspace_size: n_cells >= 1 and bytes required");
  Carver cv(nullptr);
  Ws w;
  plan(cv, w, sh, n_cells);
  *bytes = cv.off + 256;
  return JOLT_OK;
}

extern "C" int jolt_decompress_workspace_size(const jolt_cell_desc *out_desc, int n_cells, int max_rT,
                                              size_t *bytes) {
  int rc = validate_desc(out_desc);
  if (rc) return rc;
  if (n_cells < 1 || max_rT < 0 || !bytes)
    return jolt_fail(JOLT_E_INVAL, "jolt_decompress_workspace_size: n_cells >= 1, max_rT >= 0 and bytes required");
  Carver cv(nullptr);
  Ws w;
  plan_decode(cv, w, out_desc->n_layers * out_desc->n_heads, out_desc->T, out_desc->d, n_cells, max_rT);
  *bytes = cv.off + 256;
  return JOLT_OK;
}

static int check_common(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                        void *ws) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "ctx is null");
  if (n_cells < 1) return jolt_fail(JOLT_E_INVAL, "n_cells must be >= 1");
  if (!X) return jolt_fail(JOLT_E_INVAL, "X is null");
  for (int c = 0; c < n_cells; ++c) {
    if (!X[c]) return jolt_fail(JOLT_E_INVAL, "X[%d] is null", c);
    if (reinterpret_cast<uintptr_t>(X[c]) & 15) return jolt_fail(JOLT_E_INVAL, "X[%d] not 16-byte aligned", c);
  }
  if (!ws) return jolt_fail(JOLT_E_INVAL, "workspace is null");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return jolt_fail(JOLT_E_INVAL, "workspace must be 256-byte aligned");
  (void)desc;
  return JOLT_OK;
}

static bool same_desc(const jolt_cell_desc &a, const jolt_cell_desc &b) {
  return std::memcmp(&a, &b, sizeof a) == 0;
}

static bool same_opts(const jolt_spectrum_opts &a, const jolt_spectrum_opts &b) {
  return a.method == b.method && a.q == b.q && a.ratio == b.ratio && a.oversample == b.oversample &&
         a.power_iters == b.power_iters && a.r_max == b.r_max;
}

namespace {

// CholeskyQR2 of the rows x l matrices in buf (ld ldl): result back in buf, tmp is scratch.
// split (bf16 cells, whose spectra are compared at 1e-3): the products Y R^-1 and the
// second pass's Gram run on the bf16 matrix cores with both operands split into hi + lo
// (relative error ~2^-16, so the basis is orthonormal to ~1e-5 instead of fp32 accuracy).
// The first pass's Gram is always fp64: the raw range basis can be ill-conditioned, the
// first pass's output is not (its Gram has a condition number near 1).
int orth(Run &R, const SpecShape &sh, int nc, float *buf, float *tmp, int rows, bool split) {
  const int l = sh.ell, ldl = R.w.ldl;
  float *src = buf, *dst = tmp;
  for (int pass = 0; pass < 2; ++pass) {
    if (split && pass == 1) {
      // Y^T Y split over row chunks (only l x l outputs per cell: without the split too few
      // workgroups would each run the whole row loop), lower-triangle tiles, into partial
      // Grams kept in the fp64 Gram's partial area; summed in chunk order in fp64
      const int S = std::max(1, std::min({kGramSplitMax, rows / 1024, 2 * R.w.g64_chunks}));
      const int Kc = ((rows + S - 1) / S + 63) / 64 * 64;
      float *part = reinterpret_cast<float *>(R.w.g64p);
      std::vector<GemmProblem> G;
      G.reserve((size_t)nc * S);
      for (int c = 0; c < nc; ++c)
        for (int t = 0; t < S; ++t) {
          const int k0 = t * Kc, kn = std::max(0, std::min(Kc, rows - k0));
          GemmProblem p{};
          const float *y = src + (int64_t)c * rows * ldl + (int64_t)std::min(k0, rows - 1) * ldl;
          p.A = plain(y, ldl);                                       // Y^T rows chunk: m-contiguous
          p.B = plain(y, ldl);                                       // Y: n-contiguous
          p.C = part + ((int64_t)c * S + t) * l * l; p.ldc = l;
          p.M = l; p.N = l; p.K = kn; p.alpha = 1.f; p.lower_only = 1;
          G.push_back(p);
        }
      int rc = R.gemm(G, 2, GT_F32, GT_F32, false, false);
      if (rc) return rc;
      HIP_OK(launch_sum_gram_parts(part, R.w.g64, l, S, nc, R.st));
    } else {
      Gram64Args g{};
      g.Y = src; g.y_cell_stride = (int64_t)rows * ldl; g.ld = ldl;
      g.rows = rows; g.l = l; g.chunk_rows = kG64Rows; g.chunks = (rows + kG64Rows - 1) / kG64Rows;
      g.partial = R.w.g64p; g.G = R.w.g64;
      HIP_OK(launch_gram64(g, nc, R.st));
    }
    if (R.orth_calls >= kOrthMax) return jolt_fail(JOLT_E_WORKSPACE, "too many orthonormalisations");
    int32_t *clamp = R.w.orth_clamp + ((size_t)R.orth_calls * 2 + pass) * nc;
    CholArgs ca{R.w.g64, R.w.chM, R.w.Rinv, R.w.chD, R.w.chMax, clamp, l, ldl, chol_blocks(l), 0};
    HIP_OK(launch_chol_inv(ca, nc, R.st));
    std::vector<GemmProblem> P(nc);
    for (int c = 0; c < nc; ++c) {
      GemmProblem &p = P[c];
      p = GemmProblem{};
      p.A = plain(src + (int64_t)c * rows * ldl, ldl);             // k-contiguous
      p.B = plain(R.w.Rinv + (int64_t)c * l * ldl, ldl);           // n-contiguous
      p.C = dst + (int64_t)c * rows * ldl; p.ldc = ldl;
      p.M = rows; p.N = l; p.K = l; p.alpha = 1.f;
    }
    int rc = R.gemm(P, split ? 2 : 1, GT_F32, GT_F32, true, false);
    if (rc) return rc;
    std::swap(src, dst);
  }
  ++R.orth_calls;
  return JOLT_OK;
}

// FlashJoLT token spectrum: range finder with power iterations, B = Q^T X_(2), eig(B B^T)
int token_flash(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc, const void *const *X,
                const uint64_t *seeds, const jolt_spectrum_opts *o) {
  const int T = sh.T, N = sh.N, l = sh.ell, ldl = R.w.ldl, ldo = R.w.ldo;
  const int dt = dtype_gt(desc->dtype);
  HIP_OK(hipMemcpyAsync(R.w.seeds, seeds, nc * sizeof(uint64_t), hipMemcpyHostToDevice, R.st));
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_SKETCH);
    SketchArgs sa{R.w.seeds, R.w.Om, (int64_t)N * ldo, N, l, ldo, 0};
    HIP_OK(launch_sketch(sa, nc, R.st));
    std::vector<GemmProblem> P(nc);
    for (int c = 0; c < nc; ++c) {
      GemmProblem &p = P[c];
      p = GemmProblem{};
      p.A = cell_operand(X[c], desc);                               // X_(2): k-contiguous
      p.B = plain(R.w.Om + (int64_t)c * N * ldo, ldo);               // Omega: n-contiguous
      p.C = R.w.Ysk + (int64_t)c * T * ldl; p.ldc = ldl;
      p.M = T; p.N = l; p.K = N; p.alpha = 1.f;
    }
    int rc = desc->dtype == JOLT_BF16 ? R.gemm(P, 0, GT_BF16, GT_BF16, true, false)
                                      : R.gemm(P, 1, GT_F32, GT_BF16, true, false);
    if (rc) return rc;
  }
  int rc;
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_ORTH);
    rc = orth(R, sh, nc, R.w.Ysk, R.w.Qsk, T, dt == GT_BF16);
    if (rc) return rc;
  }
  for (int it = 0; it < o->power_iters; ++it) {
    std::vector<GemmProblem> P(nc);
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_SKETCH);
      for (int c = 0; c < nc; ++c) {                                 // Z = X_(2)^T Q   (N x l)
        GemmProblem &p = P[c];
        p = GemmProblem{};
        p.A = cell_operand(X[c], desc);                             // m-contiguous view of X_(2)^T
        p.B = plain(R.w.Ysk + (int64_t)c * T * ldl, ldl);
        p.C = R.w.Zsk + (int64_t)c * N * ldl; p.ldc = ldl;
        p.M = N; p.N = l; p.K = T; p.alpha = 1.f;
      }
      rc = R.gemm(P, dt == GT_BF16 ? 2 : 1, dt, GT_F32, false, false);
      if (rc) return rc;
    }
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_ORTH);
      rc = orth(R, sh, nc, R.w.Zsk, R.w.Qz, N, dt == GT_BF16);
      if (rc) return rc;
    }
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_SKETCH);
      for (int c = 0; c < nc; ++c) {                                 // Y = X_(2) Q'   (T x l)
        GemmProblem &p = P[c];
        p = GemmProblem{};
        p.A = cell_operand(X[c], desc);
        p.B = plain(R.w.Zsk + (int64_t)c * N * ldl, ldl);
        p.C = R.w.Ysk + (int64_t)c * T * ldl; p.ldc = ldl;
        p.M = T; p.N = l; p.K = N; p.alpha = 1.f;
      }
      rc = R.gemm(P, dt == GT_BF16 ? 2 : 1, dt, GT_F32, true, false);
      if (rc) return rc;
    }
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_ORTH);
      rc = orth(R, sh, nc, R.w.Ysk, R.w.Qsk, T, dt == GT_BF16);
      if (rc) return rc;
    }
  }
  {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_SKETCH);
    std::vector<GemmProblem> P(nc);
    for (int c = 0; c < nc; ++c) {                                   // B = Q^T X_(2)   (l x N)
      GemmProblem &p = P[c];
      p = GemmProblem{};
      p.A = plain(R.w.Ysk + (int64_t)c * T * ldl, ldl);              // m-contiguous view of Q^T
      p.B = cell_operand(X[c], desc);                               // n-contiguous
      p.C = R.w.Bsk + (int64_t)c * l * N; p.ldc = N;
      p.M = l; p.N = N; p.K = T; p.alpha = 1.f;
    }
    rc = R.gemm(P, dt == GT_BF16 ? 2 : 1, GT_F32, dt, false, false);
    if (rc) return rc;
    for (int c = 0; c < nc; ++c) {                                   // B B^T   (l x l)
      GemmProblem &p = P[c];
      p = GemmProblem{};
      p.A = plain(R.w.Bsk + (int64_t)c * l * N, N);
      p.B = plain(R.w.Bsk + (int64_t)c * l * N, N);
      p.C = R.w.C + (int64_t)c * l * l; p.ldc = l;
      p.M = l; p.N = l; p.K = N; p.alpha = 1.f;
    }
    rc = R.gemm(P, 1, GT_F32, GT_F32, true, true);
    if (rc) return rc;
  }
  return eig_values(R, R.w.teig);
}

int spectrum_device(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc,
                    const void *const *X, const uint64_t *seeds, const jolt_spectrum_opts *o) {
  int rc = feature_stage(R, sh, desc, nc, X);
  if (rc) return rc;
  if (sh.method == JOLT_EXACT) return token_exact(R, sh, desc, nc, X);
  return token_flash(R, sh, desc, nc, X, seeds, o);
}

}  // namespace

extern "C" int jolt_spectrum(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                             const uint64_t *seeds, const jolt_spectrum_opts *opts, void *ws,
                             size_t ws_bytes, double *E, double *lam_T, double *lam_d,
                             jolt_stream stream) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  rc = check_common(ctx, desc, n_cells, X, ws);
  if (rc) return rc;
  if (sh.method == JOLT_FLASH && !seeds) return jolt_fail(JOLT_E_INVAL, "FlashJoLT needs seeds");
  if (!E || !lam_T || !lam_d) return jolt_fail(JOLT_E_INVAL, "output arrays are null");
  size_t need = 0;
  jolt_workspace_size(desc, n_cells, opts, &need);
  if (ws_bytes < need) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  Run R{ctx, (hipStream_t)stream, {}};
  Carver cv(ws);
  plan(cv, R.w, sh, n_cells);
  forget_spectra(ctx, ws, ws_bytes);
  rc = spectrum_device(R, sh, desc, n_cells, X, seeds, opts);
  if (rc) return rc;
  std::vector<double> lt((size_t)n_cells * sh.T), ld((size_t)n_cells * sh.d);
  HIP_OK(hipMemcpyAsync(E, R.w.E, n_cells * sizeof(double), hipMemcpyDeviceToHost, R.st));
  HIP_OK(hipMemcpyAsync(ld.data(), R.w.feig.b.lam, ld.size() * sizeof(double), hipMemcpyDeviceToHost, R.st));
  std::vector<double> lf((size_t)n_cells * std::max(sh.ell, 1));
  if (sh.method == JOLT_EXACT)
    HIP_OK(hipMemcpyAsync(lt.data(), R.w.teig.b.lam, lt.size() * sizeof(double), hipMemcpyDeviceToHost, R.st));
  else
    HIP_OK(hipMemcpyAsync(lf.data(), R.w.teig.b.lam, lf.size() * sizeof(double), hipMemcpyDeviceToHost, R.st));
  CallChecks chk;
  rc = chk.queue(R, n_cells, true, false, false);
  if (rc) return rc;
  HIP_OK(hipStreamSynchronize(R.st));
  rc = chk.verdict();
  if (rc) return rc;
  // eigenvalues are clipped at 0 (the Grams are positive semi-definite)
  for (int c = 0; c < n_cells; ++c) {
    for (int i = 0; i < sh.d; ++i) lam_d[(size_t)c * sh.d + i] = std::max(0.0, ld[(size_t)c * sh.d + i]);
    if (sh.method == JOLT_EXACT) {
      for (int i = 0; i < sh.T; ++i) lam_T[(size_t)c * sh.T + i] = std::max(0.0, lt[(size_t)c * sh.T + i]);
    } else {
      // the q captured Ritz values, then the omitted energy as one synthetic value
      double captured = 0.0;
      for (int i = 0; i < sh.q; ++i) {
        const double v = std::max(0.0, lf[(size_t)c * sh.ell + i]);
        lam_T[(size_t)c * (sh.q + 1) + i] = v;
        captured += v;
      }
      lam_T[(size_t)c * (sh.q + 1) + sh.q] = std::max(0.0, E[c] - captured);
    }
  }
  ctx->specs.emplace_back();
  SpecKey &k = ctx->specs.back();
  k.valid = true;
  k.ws = ws;
  k.ws_bytes = ws_bytes;
  k.desc = *desc;
  k.opts = opts ? *opts : jolt_spectrum_opts{JOLT_EXACT, 0, 0.0, 0, 0, 0, 0};
  k.X.assign(X, X + n_cells);
  k.seeds.assign(seeds ? seeds : (const uint64_t *)nullptr, seeds ? seeds + n_cells : (const uint64_t *)nullptr);
  k.token_refl_off = R.w.teig.b.refl_off;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ compress
namespace {

// The token spectrum of these cells in the workspace: taken from it on request (the context
// must have recorded one for the same cells, options, seeds and workspace), computed and
// recorded otherwise.
int acquire_spectrum(Run &R, const SpecShape &sh, const jolt_cell_desc *desc, int nc,
                     const void *const *X, const std::vector<uint64_t> &seeds,
                     const jolt_spectrum_opts &o, void *ws, size_t ws_bytes) {
  jolt_ctx *ctx = R.ctx;
  if (o.reuse) {
    const SpecKey *found = nullptr;
    for (const SpecKey &k : ctx->specs) {
      bool ok = k.valid && k.ws == ws && k.ws_bytes == ws_bytes && same_desc(k.desc, *desc) &&
                same_opts(k.opts, o) && (int)k.X.size() == nc && std::equal(k.X.begin(), k.X.end(), X);
      if (ok && sh.method == JOLT_FLASH) ok = k.seeds == seeds;
      if (ok) { found = &k; break; }
    }
    if (!found)
      return jolt_fail(JOLT_E_STATE, "reuse requested but the workspace holds no spectrum of these cells");
    // the eigenvector back-transform follows the reduction that stored the reflectors
    R.w.teig.b.refl_off = found->token_refl_off;
    forget_spectra(ctx, ws, ws_bytes, found);
    return JOLT_OK;
  }
  forget_spectra(ctx, ws, ws_bytes);
  int rc = spectrum_device(R, sh, desc, nc, X, seeds.data(), &o);
  if (rc) return rc;
  ctx->specs.emplace_back();
  SpecKey &k = ctx->specs.back();
  k.valid = true;
  k.ws = ws;
  k.ws_bytes = ws_bytes;
  k.desc = *desc;
  k.opts = o;
  k.X.assign(X, X + nc);
  k.seeds = seeds;
  k.token_refl_off = R.w.teig.b.refl_off;
  return JOLT_OK;
}

}  // namespace

extern "C" int jolt_compress(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                             const jolt_params *params, const jolt_spectrum_opts *opts, void *ws,
                             size_t ws_bytes, void *const *blobs, const size_t *blob_bytes,
                             jolt_stream stream) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  rc = check_common(ctx, desc, n_cells, X, ws);
  if (rc) return rc;
  if (!params || !blobs || !blob_bytes) return jolt_fail(JOLT_E_INVAL, "params/blobs are null");
  for (int c = 0; c < n_cells; ++c) {
    rc = validate_params(desc, &params[c], sh.rT_max);
    if (rc) return rc;
    if (params[c].group != params[0].group || params[c].factor_dtype != params[0].factor_dtype)
      return jolt_fail(JOLT_E_INVAL, "group and factor_dtype must be equal across the cells of a call");
    size_t need = 0;
    jolt_compressed_size(desc, &params[c], &need);
    if (!blobs[c] || blob_bytes[c] < need)
      return jolt_fail(JOLT_E_WORKSPACE, "blob %d: %zu bytes < %zu", c, blob_bytes[c], need);
    if (reinterpret_cast<uintptr_t>(blobs[c]) & 255) return jolt_fail(JOLT_E_INVAL, "blob %d not 256-byte aligned", c);
  }
  size_t need = 0;
  jolt_workspace_size(desc, n_cells, opts, &need);
  if (ws_bytes < need) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  Run R{ctx, (hipStream_t)stream, {}};
  Carver cv(ws);
  plan(cv, R.w, sh, n_cells);
  const int m = sh.m, T = sh.T, d = sh.d, N = sh.N, nc = n_cells;
  std::vector<uint64_t> seeds(nc);
  for (int c = 0; c < nc; ++c) seeds[c] = params[c].seed;
  jolt_spectrum_opts o = opts ? *opts : jolt_spectrum_opts{JOLT_EXACT, 0, 0.0, 0, 0, 0, 0};
  rc = acquire_spectrum(R, sh, desc, nc, X, seeds, o, ws, ws_bytes);
  if (rc) return rc;
  rc = upload_seeds_and_signs(R, seeds.data(), nc, d);
  if (rc) return rc;
  std::vector<int> rT(nc), rd(nc);
  int kmax = 0;
  for (int c = 0; c < nc; ++c) { rT[c] = params[c].r_T; rd[c] = params[c].r_d; kmax = std::max(kmax, rT[c]); }
  const int64_t ldu = R.w.kmaxT, u_stride = (int64_t)T * R.w.kmaxT;
  const int64_t y_stride = (int64_t)R.w.kmaxT * N;
  const int64_t g_stride = (int64_t)m * R.w.kmaxT * d, g_slice = (int64_t)R.w.kmaxT * d;
  const bool f16 = params[0].factor_dtype == JOLT_FACTOR_F16;
  const int fb = f16 ? 2 : 4, ft = f16 ? GT_F16 : GT_F32;
  std::vector<BlobLayout> L(nc);
  for (int c = 0; c < nc; ++c) L[c] = blob_layout(m, T, d, rT[c], rd[c], params[c].bits, params[0].group, fb);
  if (kmax > 0) {
    std::vector<GemmProblem> P;
    if (sh.method == JOLT_EXACT) {
      // token factor U_T: top r_T eigenvectors of the token Gram
      rc = eig_vectors(R, R.w.teig, rT, R.w.U, ldu, u_stride);
      if (rc) return rc;
      // Y = U_T^T X_(2)   (r_T x N per cell)
      for (int c = 0; c < nc; ++c) {
        if (!rT[c]) continue;
        GemmProblem p{};
        p.A = plain(R.w.U + c * u_stride, ldu);        // A(m = r, k = t) = U[t][r]: m-contiguous
        p.B = cell_operand(X[c], desc);                // B(k = t, n = col): n-contiguous
        p.C = R.w.Y + c * y_stride; p.ldc = N;
        p.M = rT[c]; p.N = N; p.K = T; p.alpha = 1.f;
        P.push_back(p);
      }
      StageTimer t(R.ctx, R.st, JOLT_STAGE_PROJECT);
      rc = R.gemm(P, desc->dtype == JOLT_BF16 ? 2 : 1, GT_F32, dtype_gt(desc->dtype), false, false);
      if (rc) return rc;
    } else {
      // FlashJoLT: Ritz vectors W of B B^T, U_T = Q W, and Y = W_r^T B (no pass over X)
      const int l = sh.ell, q = sh.q, ldl = R.w.ldl;
      rc = eig_vectors(R, R.w.teig, rT, R.w.Wsk, q, (int64_t)l * q);
      if (rc) return rc;
      StageTimer t(R.ctx, R.st, JOLT_STAGE_PROJECT);
      for (int c = 0; c < nc; ++c) {
        if (!rT[c]) continue;
        GemmProblem p{};
        p.A = plain(R.w.Ysk + (int64_t)c * T * ldl, ldl);             // Q: k-contiguous
        p.B = plain(R.w.Wsk + (int64_t)c * l * q, q);                 // W: n-contiguous
        p.C = R.w.U + c * u_stride; p.ldc = ldu;
        p.M = T; p.N = rT[c]; p.K = l; p.alpha = 1.f;
        P.push_back(p);
      }
      rc = R.gemm(P, 1, GT_F32, GT_F32, true, false);
      if (rc) return rc;
      P.clear();
      for (int c = 0; c < nc; ++c) {
        if (!rT[c]) continue;
        GemmProblem p{};
        p.A = plain(R.w.Wsk + (int64_t)c * l * q, q);                 // W^T: m-contiguous
        p.B = plain(R.w.Bsk + (int64_t)c * l * N, N);                 // B: n-contiguous
        p.C = R.w.Y + c * y_stride; p.ldc = N;
        p.M = rT[c]; p.N = N; p.K = l; p.alpha = 1.f;
        P.push_back(p);
      }
      rc = R.gemm(P, 1, GT_F32, GT_F32, false, false);
      if (rc) return rc;
    }
    // feature factor from the Gram of Y: F_Y = sum_s Y_s^T Y_s, top r_d eigenvectors
    std::vector<FGramCell> fc(nc);
    for (int c = 0; c < nc; ++c) fc[c] = FGramCell{R.w.Y + c * y_stride, rT[c], 0};
    HIP_OK(hipMemcpyAsync(R.w.fcell, fc.data(), nc * sizeof(FGramCell), hipMemcpyHostToDevice, R.st));
    FGramArgs a{};
    a.cells = R.w.fcell; a.n_cells = nc; a.nseg = m; a.seg_heads = 1; a.seg_hi = d; a.seg_lo = 0;
    a.row_stride = N; a.chunks_per_cell = R.w.chunks; a.partial_F = R.w.fpart; a.partial_E = R.w.epart;
    a.nonfinite = R.w.nonfinite;
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_FEATURE_GRAM);
      HIP_OK(launch_feature_gram(a, d, JOLT_F32, R.st));
      HIP_OK(launch_feature_gram_reduce(a, d, R.w.F, R.w.E, R.st));
    }
    rc = eig_values(R, R.w.feig);
    if (rc) return rc;
    rc = eig_vectors(R, R.w.feig, rd, R.w.Ud, d, (int64_t)d * d);
    if (rc) return rc;
    // core G_s = Y_s U_d   (r_T x r_d per slice)
    P.clear();
    for (int c = 0; c < nc; ++c) {
      if (!rT[c]) continue;
      for (int s = 0; s < m; ++s) {
        GemmProblem p{};
        p.A = plain(R.w.Y + c * y_stride + (int64_t)s * d, N);     // k-contiguous
        p.B = plain(R.w.Ud + (int64_t)c * d * d, d);               // n-contiguous
        p.C = R.w.G + c * g_stride + s * g_slice; p.ldc = d;
        p.M = rT[c]; p.N = rd[c]; p.K = d; p.alpha = 1.f;
        P.push_back(p);
      }
    }
    {
      StageTimer t(R.ctx, R.st, JOLT_STAGE_CORE);
      rc = R.gemm(P, 1, GT_F32, GT_F32, true, false);
      if (rc) return rc;
    }
    // serialise U_T, U_d, G (fp16 with per-slice exponents, or fp32)
    std::vector<SerFactorCell> sf(2 * nc);
    std::vector<SerCell> sc(nc);
    int64_t maxel = 0;
    for (int c = 0; c < nc; ++c) {
      uint8_t *b = static_cast<uint8_t *>(blobs[c]);
      sf[c] = SerFactorCell{R.w.U + c * u_stride, ldu, b + L[c].UT, T, rT[c], f16 ? 1 : 0, 0};
      sf[nc + c] = SerFactorCell{R.w.Ud + (int64_t)c * d * d, d, b + L[c].Ud, d, rd[c], f16 ? 1 : 0, 0};
      sc[c] = SerCell{R.w.G + c * g_stride, g_slice, d, b + L[c].G, reinterpret_cast<int8_t *>(b + L[c].gexp),
                      rT[c], rd[c], f16 ? 1 : 0, 0};
      maxel = std::max<int64_t>(maxel, (int64_t)T * rT[c]);
    }
    HIP_OK(hipMemcpyAsync(R.w.sfcell, sf.data(), sf.size() * sizeof(SerFactorCell), hipMemcpyHostToDevice, R.st));
    HIP_OK(hipMemcpyAsync(R.w.scell, sc.data(), sc.size() * sizeof(SerCell), hipMemcpyHostToDevice, R.st));
    StageTimer t(R.ctx, R.st, JOLT_STAGE_SERIALIZE);
    HIP_OK(launch_factor_pack(SerFactor{R.w.sfcell}, 2 * nc, maxel, R.st));
    HIP_OK(launch_core_pack(SerCore{R.w.scell, m}, nc, R.st));
  }
  // zero exponents of cells without a backbone (the section is still present)
  for (int c = 0; c < nc; ++c)
    if (!rT[c]) HIP_OK(hipMemsetAsync(static_cast<uint8_t *>(blobs[c]) + L[c].gexp, 0, m, R.st));
  // residual against X~ = U^_T W_s rebuilt from the stored factors inside the fused pass:
  // W_s^T and its exponents first, then reconstruction + rotation + quantisation + packing
  std::vector<BlobView> bv(nc);
  std::vector<FusedCell> fc(nc);
  bool any_bits = false;
  for (int c = 0; c < nc; ++c) {
    bv[c] = BlobView{static_cast<const uint8_t *>(blobs[c]), L[c], rT[c], rd[c], params[c].bits};
    fc[c] = fused_cell(R, c, m, d, bv[c]);
    fc[c].x = X[c];
    any_bits |= params[c].bits != 0;
  }
  if (kmax > 0) {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_RECONSTRUCT);
    rc = build_w(R, nc, m, d, bv, fc, fb);
    if (rc) return rc;
  } else {
    HIP_OK(hipMemcpyAsync(R.w.fcell_r, fc.data(), nc * sizeof(FusedCell), hipMemcpyHostToDevice, R.st));
  }
  if (any_bits) {
    StageTimer t(R.ctx, R.st, JOLT_STAGE_RESIDUAL);
    HIP_OK(launch_fused(fused_args(R, nc, m, T, d, params[0].group, desc), FUSED_RESIDUAL, d, desc->dtype,
                        !f16, R.st));
  }
  // headers
  std::vector<uint8_t> hdr((size_t)nc * kHeaderBytes);
  for (int c = 0; c < nc; ++c) {
    fill_header(hdr.data() + (size_t)c * kHeaderBytes, desc, &params[c], sh.method);
    HIP_OK(hipMemcpyAsync(blobs[c], hdr.data() + (size_t)c * kHeaderBytes, kHeaderBytes, hipMemcpyHostToDevice, R.st));
  }
  // input and solver checks (a spectrum computed here; the eigenvectors of this call)
  CallChecks chk;
  rc = chk.queue(R, nc, !o.reuse, kmax > 0, kmax > 0);
  if (rc) return rc;
  HIP_OK(hipStreamSynchronize(R.st));
  rc = chk.verdict();
  if (rc) {
    forget_spectra(ctx, ws, ws_bytes);
    return rc;
  }
  DebugState &dbg = ctx->dbg;
  dbg.valid = true;
  dbg.n_cells = nc; dbg.T = T; dbg.d = d; dbg.m = m; dbg.N = N; dbg.ell = sh.ell;
  dbg.rT = rT; dbg.rd = rd;
  dbg.U = R.w.U; dbg.u_stride = u_stride; dbg.ldu = ldu;
  dbg.Ud = R.w.Ud; dbg.ud_stride = (int64_t)d * d;
  // the X~ export re-runs the fused pass in its export mode on this call's W_s^T
  dbg.fused = fc;
  dbg.fcell_dev = R.w.fcell_r;
  dbg.fargs = fused_args(R, nc, m, T, d, params[0].group, desc);
  dbg.split = !f16;
  dbg.Omega = R.w.Om; dbg.om_stride = (int64_t)N * R.w.ldo; dbg.ldo = R.w.ldo;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ truncated feature spectra
namespace {

struct TruncWs {
  GemmProblem *tab = nullptr;   // replaces the spectrum plan's table for this call
  size_t tab_n = 0;
  FGramCell *fcell = nullptr;   // one per (cell, row block)
  double *epart = nullptr;
  int32_t *nonfinite = nullptr;
  float *F = nullptr;           // [cell][block][d][d]: block Grams, then running sums
  EigWs eig;
};

void plan_trunc(Carver &cv, TruncWs &t, const Ws &w, int nc, int n_r, int d) {
  const size_t nm = (size_t)nc * n_r;
  t.tab_n = w.tab_n + 2 * (size_t)nc;
  t.tab = cv.take<GemmProblem>(t.tab_n);
  t.fcell = cv.take<FGramCell>(nm);
  t.epart = cv.take<double>(nm);
  t.nonfinite = cv.take<int32_t>(nm);
  t.F = cv.take<float>(nm * d * d);
  carve_eig(cv, t.eig, (int)nm, d, 0, t.F);
}

int check_trunc(const SpecShape &sh, int step, int n_r) {
  if (step < 1 || n_r < 1 || (int64_t)step * n_r > sh.rT_max)
    return jolt_fail(JOLT_E_INVAL, "step %d x n_r %d must be >= 1 and <= rT_max %d", step, n_r, sh.rT_max);
  return JOLT_OK;
}

}  // namespace

extern "C" int jolt_truncated_spectra_workspace_size(const jolt_cell_desc *desc, int n_cells,
                                                     const jolt_spectrum_opts *opts, int step, int n_r,
                                                     size_t *bytes) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  rc = check_trunc(sh, step, n_r);
  if (rc) return rc;
  if (n_cells < 1 || !bytes) return jolt_fail(JOLT_E_INVAL, "n_cells >= 1 and bytes required");
  Carver cv(nullptr);
  Ws w;
  plan(cv, w, sh, n_cells);
  TruncWs t;
  plan_trunc(cv, t, w, n_cells, n_r, sh.d);
  *bytes = cv.off;
  return JOLT_OK;
}

extern "C" int jolt_truncated_spectra(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells,
                                      const void *const *X, const uint64_t *seeds,
                                      const jolt_spectrum_opts *opts, int step, int n_r, void *ws,
                                      size_t ws_bytes, double *mu, jolt_stream stream) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  rc = check_trunc(sh, step, n_r);
  if (rc) return rc;
  rc = check_common(ctx, desc, n_cells, X, ws);
  if (rc) return rc;
  if (sh.method == JOLT_FLASH && !seeds) return jolt_fail(JOLT_E_INVAL, "FlashJoLT needs seeds");
  if (!mu) return jolt_fail(JOLT_E_INVAL, "mu is null");
  size_t need = 0;
  jolt_truncated_spectra_workspace_size(desc, n_cells, opts, step, n_r, &need);
  if (ws_bytes < need) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  Run R{ctx, (hipStream_t)stream, {}};
  Carver cv(ws);
  plan(cv, R.w, sh, n_cells);
  TruncWs t;
  plan_trunc(cv, t, R.w, n_cells, n_r, sh.d);
  R.w.tab = t.tab;
  R.w.tab_n = t.tab_n;
  const int m = sh.m, T = sh.T, d = sh.d, N = sh.N, nc = n_cells, rmax = step * n_r;
  std::vector<uint64_t> sd(nc, 0);
  if (seeds) std::copy(seeds, seeds + nc, sd.begin());
  jolt_spectrum_opts o = opts ? *opts : jolt_spectrum_opts{JOLT_EXACT, 0, 0.0, 0, 0, 0, 0};
  rc = acquire_spectrum(R, sh, desc, nc, X, sd, o, ws, ws_bytes);
  if (rc) return rc;
  // Y = U_r^T X_(2) at r = n_r * step (rows r, columns s * d + f), as the compression's
  // projection forms it
  const std::vector<int> kr(nc, rmax);
  const int64_t ldu = R.w.kmaxT, u_stride = (int64_t)T * R.w.kmaxT, y_stride = (int64_t)R.w.kmaxT * N;
  std::vector<GemmProblem> P;
  if (sh.method == JOLT_EXACT) {
    rc = eig_vectors(R, R.w.teig, kr, R.w.U, ldu, u_stride);
    if (rc) return rc;
    for (int c = 0; c < nc; ++c) {
      GemmProblem p{};
      p.A = plain(R.w.U + c * u_stride, ldu);
      p.B = cell_operand(X[c], desc);
      p.C = R.w.Y + c * y_stride; p.ldc = N;
      p.M = rmax; p.N = N; p.K = T; p.alpha = 1.f;
      P.push_back(p);
    }
    StageTimer tm(R.ctx, R.st, JOLT_STAGE_PROJECT);
    rc = R.gemm(P, desc->dtype == JOLT_BF16 ? 2 : 1, GT_F32, dtype_gt(desc->dtype), false, false);
    if (rc) return rc;
  } else {
    const int l = sh.ell, q = sh.q;
    rc = eig_vectors(R, R.w.teig, kr, R.w.Wsk, q, (int64_t)l * q);
    if (rc) return rc;
    for (int c = 0; c < nc; ++c) {
      GemmProblem p{};
      p.A = plain(R.w.Wsk + (int64_t)c * l * q, q);
      p.B = plain(R.w.Bsk + (int64_t)c * l * N, N);
      p.C = R.w.Y + c * y_stride; p.ldc = N;
      p.M = rmax; p.N = N; p.K = l; p.alpha = 1.f;
      P.push_back(p);
    }
    StageTimer tm(R.ctx, R.st, JOLT_STAGE_PROJECT);
    rc = R.gemm(P, 1, GT_F32, GT_F32, false, false);
    if (rc) return rc;
  }
  // Gram of every row block k of Y (rows k step .. (k+1) step - 1 of all m slices), then
  // running sums over k: F_Y((k+1) step)
  const int nm = nc * n_r;
  std::vector<FGramCell> fc(nm);
  for (int c = 0; c < nc; ++c)
    for (int k = 0; k < n_r; ++k) fc[(size_t)c * n_r + k] = FGramCell{R.w.Y + c * y_stride + (int64_t)k * step * N, step, 0};
  HIP_OK(hipMemcpyAsync(t.fcell, fc.data(), nm * sizeof(FGramCell), hipMemcpyHostToDevice, R.st));
  FGramArgs a{};
  a.cells = t.fcell; a.n_cells = nm; a.nseg = m; a.seg_heads = 1; a.seg_hi = d; a.seg_lo = 0;
  a.row_stride = N; a.chunks_per_cell = 1; a.partial_F = t.F; a.partial_E = t.epart;
  a.nonfinite = t.nonfinite;
  {
    StageTimer tm(R.ctx, R.st, JOLT_STAGE_TRUNC_GRAM);
    HIP_OK(launch_feature_gram(a, d, JOLT_F32, R.st));
    HIP_OK(launch_prefix_sum_mats(t.F, nc, n_r, (int64_t)d * d, R.st));
  }
  rc = eig_values(R, t.eig);
  if (rc) return rc;
  HIP_OK(hipMemcpyAsync(mu, t.eig.b.lam, (size_t)nm * d * sizeof(double), hipMemcpyDeviceToHost, R.st));
  CallChecks chk;
  rc = chk.queue(R, nc, !o.reuse, true, false);
  if (rc) return rc;
  HIP_OK(hipStreamSynchronize(R.st));
  rc = chk.verdict();
  if (rc) {
    forget_spectra(ctx, ws, ws_bytes);
    return rc;
  }
  for (size_t i = 0; i < (size_t)nm * d; ++i) mu[i] = std::max(0.0, mu[i]);
  return JOLT_OK;
}

// ------------------------------------------------------------------------ decompress
extern "C" int jolt_decompress(jolt_ctx *ctx, int n_cells, const void *const *blobs, const size_t *blob_bytes,
                               const void *hdr_host, const jolt_cell_desc *out, void *const *Xhat, void *ws,
                               size_t ws_bytes, jolt_stream stream) {
  return jolt_decompress_rope(ctx, n_cells, blobs, blob_bytes, hdr_host, out, Xhat, nullptr, ws, ws_bytes,
                              stream);
}

extern "C" int jolt_decompress_rope(jolt_ctx *ctx, int n_cells, const void *const *blobs,
                                    const size_t *blob_bytes, const void *hdr_host, const jolt_cell_desc *out,
                                    void *const *Xhat, const jolt_rope *rope, void *ws, size_t ws_bytes,
                                    jolt_stream stream) {
  int rc = validate_desc(out);
  if (rc) return rc;
  if (rope && (!(rope->base > 1.0) || rope->position_offset < 0))
    return jolt_fail(JOLT_E_INVAL, "jolt_decompress_rope: base must be > 1 and position_offset >= 0");
  if (n_cells < 1 || !blobs || !blob_bytes || !Xhat || !ws)
    return jolt_fail(JOLT_E_INVAL, "jolt_decompress: null argument");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return jolt_fail(JOLT_E_INVAL, "workspace must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  DeviceGuard dg;
  std::vector<uint8_t> hdr((size_t)n_cells * kHeaderBytes);
  if (hdr_host) {
    // host header copies are validated before the context is touched
    std::memcpy(hdr.data(), hdr_host, hdr.size());
    for (int c = 0; c < n_cells; ++c) {
      BlobInfo tmp;
      rc = parse_header(hdr.data() + (size_t)c * kHeaderBytes, blob_bytes[c], &tmp);
      if (rc) return rc;
    }
    if (!ctx) return jolt_fail(JOLT_E_INVAL, "jolt_decompress: ctx is null");
    HIP_OK(dg.enter(ctx->device));
  } else {
    if (!ctx) return jolt_fail(JOLT_E_INVAL, "jolt_decompress: ctx is null");
    HIP_OK(dg.enter(ctx->device));
    for (int c = 0; c < n_cells; ++c) {
      if (!blobs[c] || blob_bytes[c] < (size_t)kHeaderBytes) return jolt_fail(JOLT_E_BLOB, "blob %d too small", c);
      HIP_OK(hipMemcpyAsync(hdr.data() + (size_t)c * kHeaderBytes, blobs[c], kHeaderBytes, hipMemcpyDeviceToHost, st));
    }
    HIP_OK(hipStreamSynchronize(st));
  }
  const int m = out->n_layers * out->n_heads, T = out->T, d = out->d, N = m * d;
  std::vector<BlobInfo> bi(n_cells);
  int kmax = 0;
  for (int c = 0; c < n_cells; ++c) {
    if (!blobs[c] || !Xhat[c]) return jolt_fail(JOLT_E_INVAL, "blob/Xhat %d is null", c);
    if (reinterpret_cast<uintptr_t>(Xhat[c]) & 15) return jolt_fail(JOLT_E_INVAL, "Xhat[%d] not 16-byte aligned", c);
    rc = parse_header(hdr.data() + (size_t)c * kHeaderBytes, blob_bytes[c], &bi[c]);
    if (rc) return rc;
    const BlobInfo &b = bi[c];
    if ((int)b.m != m || (int)b.T != T || (int)b.d != d || (int)b.heads != out->n_heads)
      return jolt_fail(JOLT_E_BLOB, "blob %d shape (m %u, T %u, d %u) differs from the output descriptor", c, b.m, b.T, b.d);
    if (b.group != bi[0].group || b.f16 != bi[0].f16)
      return jolt_fail(JOLT_E_BLOB, "group and factor precision must be equal across the blobs of a call");
    if ((int)b.rT > std::min(T, N) || (int)b.rd > d || (b.rT == 0) != (b.rd == 0) || d % b.group || b.group % 8)
      return jolt_fail(JOLT_E_BLOB, "blob %d has invalid ranks or group", c);
    kmax = std::max(kmax, (int)b.rT);
  }
  Run R{ctx, st, {}};
  {
    Carver cv(nullptr);
    Ws w;
    plan_decode(cv, w, m, T, d, n_cells, kmax);
    if (ws_bytes < cv.off) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, cv.off);
  }
  forget_spectra(ctx, ws, ws_bytes);
  Carver cv(ws);
  plan_decode(cv, R.w, m, T, d, n_cells, kmax);
  std::vector<uint64_t> seeds(n_cells);
  for (int c = 0; c < n_cells; ++c) seeds[c] = bi[c].seed;
  rc = upload_seeds_and_signs(R, seeds.data(), n_cells, d);
  if (rc) return rc;
  const int fb = bi[0].f16 ? 2 : 4;
  // X^ = X~ + unrotated residual, X~ = U^_T W_s rebuilt inside the fused decode pass
  std::vector<BlobView> bv(n_cells);
  std::vector<FusedCell> fc(n_cells);
  for (int c = 0; c < n_cells; ++c) {
    const BlobInfo &b = bi[c];
    bv[c] = BlobView{static_cast<const uint8_t *>(blobs[c]), b.L, (int)b.rT, (int)b.rd, (int)b.bits};
    fc[c] = fused_cell(R, c, m, d, bv[c]);
    fc[c].out = Xhat[c];
  }
  if (kmax > 0) {
    StageTimer t(ctx, st, JOLT_STAGE_RECONSTRUCT);
    rc = build_w(R, n_cells, m, d, bv, fc, fb);
    if (rc) return rc;
  } else {
    HIP_OK(hipMemcpyAsync(R.w.fcell_r, fc.data(), n_cells * sizeof(FusedCell), hipMemcpyHostToDevice, st));
  }
  FusedArgs a = fused_args(R, n_cells, m, T, d, bi[0].group, out);
  if (rope) {
    a.rope = 1;
    a.rope_offset = rope->position_offset;
    a.rope_log2_base = std::log2(rope->base);
  }
  StageTimer t(ctx, st, JOLT_STAGE_DECODE);
  HIP_OK(launch_fused(a, FUSED_DECODE, d, out->dtype, !bi[0].f16, st));
  return JOLT_OK;
}

// ------------------------------------------------------------------------ eps^2 calibration
extern "C" int jolt_eps2_workspace_size(int d, int n_samples, size_t *bytes) {
  if (!bytes || (d != 32 && d != 64 && d != 128) || n_samples < d || n_samples % d)
    return jolt_fail(JOLT_E_INVAL, "jolt_eps2_workspace_size: d in {32,64,128}, n_samples a positive multiple of d");
  *bytes = (size_t)eps2_blocks() * 4 * sizeof(double) + 256;
  return JOLT_OK;
}

extern "C" int jolt_eps2_calibrate(jolt_ctx *ctx, int group, int d, uint64_t seed, int n_samples,
                                   double eps2_out[4], void *ws, size_t ws_bytes, jolt_stream stream) {
  size_t need = 0;
  int rc = jolt_eps2_workspace_size(d, n_samples, &need);
  if (rc) return rc;
  if (!ctx || !eps2_out || !ws) return jolt_fail(JOLT_E_INVAL, "jolt_eps2_calibrate: null argument");
  if (group < 8 || group > d || d % group || group % 8) return jolt_fail(JOLT_E_INVAL, "bad group %d", group);
  if (ws_bytes < need) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  forget_spectra(ctx, ws, ws_bytes);
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  hipStream_t st = (hipStream_t)stream;
  Eps2Args a{seed, n_samples, group, (float)(1.0 / std::sqrt((double)d)), static_cast<double *>(ws)};
  HIP_OK(launch_eps2_partial(a, d, st));
  std::vector<double> part((size_t)eps2_blocks() * 4);
  HIP_OK(hipMemcpyAsync(part.data(), ws, part.size() * sizeof(double), hipMemcpyDeviceToHost, st));
  HIP_OK(hipStreamSynchronize(st));
  double s[4] = {0, 0, 0, 0};
  for (int b = 0; b < eps2_blocks(); ++b)
    for (int k = 0; k < 4; ++k) s[k] += part[(size_t)b * 4 + k];
  eps2_out[0] = 1.0;
  for (int k = 1; k < 4; ++k) eps2_out[k] = s[0] > 0 ? s[k] / s[0] : 0.0;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ slice-mode spectrum
namespace {
constexpr int kSliceTileRows = 16;

int slice_chunks(int T) { return std::max(1, std::min(256, (T + 63) / 64)); }

// workspace: cell table, fp64 partials, the fp32 Gram and the eigensolver arrays
void plan_slice(Carver &cv, int m, int T, int nc, FGramCell **cells, double **partial, EigWs &e) {
  *cells = cv.take<FGramCell>(nc);
  *partial = cv.take<double>((size_t)nc * slice_chunks(T) * m * m);
  float *S = cv.take<float>((size_t)nc * m * m);
  carve_eig(cv, e, nc, m, 0, S);
}
}  // namespace

extern "C" int jolt_slice_spectrum_workspace_size(const jolt_cell_desc *desc, int n_cells, size_t *bytes) {
  if (!bytes || n_cells < 1) return jolt_fail(JOLT_E_INVAL, "jolt_slice_spectrum_workspace_size: bad argument");
  int rc = validate_desc(desc);
  if (rc) return rc;
  const int m = desc->n_layers * desc->n_heads;
  if (m > SYTRD_SMALL_MAX) return jolt_fail(JOLT_E_UNSUPPORTED, "slice spectrum limited to m <= %d", SYTRD_SMALL_MAX);
  Carver cv(nullptr);
  FGramCell *fc;
  double *part;
  EigWs e;
  plan_slice(cv, m, desc->T, n_cells, &fc, &part, e);
  *bytes = cv.off + 256;
  return JOLT_OK;
}

extern "C" int jolt_slice_spectrum(jolt_ctx *ctx, const jolt_cell_desc *desc, int n_cells, const void *const *X,
                                   void *ws, size_t ws_bytes, double *lam_s, jolt_stream stream) {
  size_t need = 0;
  int rc = jolt_slice_spectrum_workspace_size(desc, n_cells, &need);
  if (rc) return rc;
  rc = check_common(ctx, desc, n_cells, X, ws);
  if (rc) return rc;
  if (!lam_s) return jolt_fail(JOLT_E_INVAL, "lam_s is null");
  if (ws_bytes < need) return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  forget_spectra(ctx, ws, ws_bytes);
  hipStream_t st = (hipStream_t)stream;
  const int m = desc->n_layers * desc->n_heads;
  Carver cv(ws);
  FGramCell *fc;
  double *part;
  EigWs e;
  plan_slice(cv, m, desc->T, n_cells, &fc, &part, e);
  std::vector<FGramCell> cells(n_cells);
  for (int c = 0; c < n_cells; ++c) cells[c] = FGramCell{X[c], desc->T, 0};
  HIP_OK(hipMemcpyAsync(fc, cells.data(), n_cells * sizeof(FGramCell), hipMemcpyHostToDevice, st));
  SliceGramArgs a{};
  a.cells = fc;
  a.n_cells = n_cells; a.m = m; a.T = desc->T; a.heads = desc->n_heads;
  a.s_layer = desc->stride_layer; a.s_head = desc->stride_head; a.s_tok = desc->stride_token;
  a.tiles = (m + kSliceTileRows - 1) / kSliceTileRows;
  a.chunks = slice_chunks(desc->T);
  a.partial = part;
  {
    StageTimer t(ctx, st, JOLT_STAGE_SLICE_GRAM);
    HIP_OK(launch_slice_gram(a, desc->d, desc->dtype, st));
    HIP_OK(launch_slice_gram_reduce(a, e.b.A, st));
  }
  {
    StageTimer t(ctx, st, JOLT_STAGE_TRIDIAG_SMALL);
    HIP_OK(launch_sytrd_small(e.b, st));
  }
  {
    StageTimer t(ctx, st, JOLT_STAGE_EIGVALS);
    HIP_OK(launch_tridiag_eigvals(e.b, st));
  }
  std::vector<double> lam((size_t)n_cells * m);
  HIP_OK(hipMemcpyAsync(lam.data(), e.b.lam, lam.size() * sizeof(double), hipMemcpyDeviceToHost, st));
  HIP_OK(hipStreamSynchronize(st));
  // eigenvalues are clipped at 0 (the Gram is positive semi-definite)
  for (size_t i = 0; i < lam.size(); ++i) lam_s[i] = std::max(0.0, lam[i]);
  return JOLT_OK;
}

// ------------------------------------------------------------------------ attention on the factors
namespace {
void plan_attend(Carver &cv, int n, int n_q, int T, int d, int rk, int rv, AttnItem **items, uint64_t **seeds,
                 float **signs, float **gk, float **qr, float **part) {
  const int chunks = (T + ATTN_CHUNK - 1) / ATTN_CHUNK;
  *items = cv.take<AttnItem>(n);
  *seeds = cv.take<uint64_t>(2 * (size_t)n);
  *signs = cv.take<float>(2 * (size_t)n * d);
  *gk = cv.take<float>((size_t)n * n_q * std::max(rk, 1));
  *qr = cv.take<float>((size_t)n * n_q * d);
  *part = cv.take<float>((size_t)n * chunks * n_q * (2 + rv + d));
}
}  // namespace

extern "C" int jolt_attend_workspace_size(int n_items, int n_q, int T, int d, int max_rT_k, int max_rT_v,
                                          size_t *bytes) {
  if (!bytes || n_items < 1 || n_q < 1 || T < 1 || (d != 32 && d != 64 && d != 128) || max_rT_k < 0 ||
      max_rT_v < 0 || max_rT_k > ATTN_RT_MAX || max_rT_v > ATTN_RT_MAX)
    return jolt_fail(JOLT_E_INVAL, "jolt_attend_workspace_size: bad argument (ranks <= %d)", ATTN_RT_MAX);
  Carver cv(nullptr);
  AttnItem *it; uint64_t *sd; float *sg, *gk, *qr, *part;
  plan_attend(cv, n_items, n_q, T, d, max_rT_k, max_rT_v, &it, &sd, &sg, &gk, &qr, &part);
  *bytes = cv.off + 256;
  return JOLT_OK;
}

namespace {
// Decode attention on the factors with the workspace ws; caller_ws: the caller owns ws (a
// recorded spectrum it overlaps is dropped), otherwise ws is the library's fixed scratch.
int attend_impl(jolt_ctx *ctx, int n_items, const void *const *k_blobs, const size_t *k_bytes,
                const void *const *v_blobs, const size_t *v_bytes, const void *k_hdr_host,
                const void *v_hdr_host, const int32_t *layers, int n_q, const float *Q, float scale,
                float *O, void *ws, size_t ws_bytes, bool caller_ws, jolt_stream stream) {
  if (!ctx || n_items < 1 || !k_blobs || !k_bytes || !v_blobs || !v_bytes || !k_hdr_host || !v_hdr_host ||
      !layers || n_q < 1 || !Q || !O || !ws)
    return jolt_fail(JOLT_E_INVAL, "jolt_attend: null argument or empty call");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return jolt_fail(JOLT_E_INVAL, "workspace must be 256-byte aligned");
  if (!(scale > 0.f) || !std::isfinite(scale)) return jolt_fail(JOLT_E_INVAL, "jolt_attend: scale must be > 0");
  const uint8_t *kh = static_cast<const uint8_t *>(k_hdr_host), *vh = static_cast<const uint8_t *>(v_hdr_host);
  std::vector<BlobInfo> kb(n_items), vb(n_items);
  int rk = 0, rv = 0;
  for (int i = 0; i < n_items; ++i) {
    int rc = parse_header(kh + (size_t)i * kHeaderBytes, k_bytes[i], &kb[i]);
    if (rc) return rc;
    rc = parse_header(vh + (size_t)i * kHeaderBytes, v_bytes[i], &vb[i]);
    if (rc) return rc;
    const BlobInfo &a = kb[i], &b = vb[i], &z = kb[0];
    if (a.m != b.m || a.T != b.T || a.d != b.d || a.heads != b.heads || a.group != b.group)
      return jolt_fail(JOLT_E_BLOB, "item %d: key and value blobs differ in shape or group", i);
    if (a.T != z.T || a.d != z.d || a.heads != z.heads || a.group != z.group || a.m != z.m)
      return jolt_fail(JOLT_E_BLOB, "item %d: all items of a call must share m, T, d, heads and group", i);
    if (!k_blobs[i] || !v_blobs[i]) return jolt_fail(JOLT_E_INVAL, "item %d: null blob", i);
    if (layers[i] < 0 || (int64_t)layers[i] * a.heads >= a.m)
      return jolt_fail(JOLT_E_INVAL, "item %d: layer %d outside the cell's %u layers", i, layers[i], a.m / a.heads);
    if ((int)a.rT > ATTN_RT_MAX || (int)b.rT > ATTN_RT_MAX)
      return jolt_fail(JOLT_E_UNSUPPORTED, "jolt_attend: ranks above %d", ATTN_RT_MAX);
    rk = std::max(rk, (int)a.rT);
    rv = std::max(rv, (int)b.rT);
  }
  const int T = kb[0].T, d = kb[0].d, H = kb[0].heads;
  if (T > 8192 * ATTN_CHUNK) return jolt_fail(JOLT_E_UNSUPPORTED, "jolt_attend: T above %d", 8192 * ATTN_CHUNK);
  if (n_q % H) return jolt_fail(JOLT_E_INVAL, "jolt_attend: n_q = %d is not a multiple of the %d key-value heads", n_q, H);
  if (n_q > ATTN_QMAX || n_q / H > ATTN_REP_MAX)
    return jolt_fail(JOLT_E_UNSUPPORTED, "jolt_attend: at most %d query heads, %d per key-value head", ATTN_QMAX, ATTN_REP_MAX);
  size_t need = 0;
  int rc = jolt_attend_workspace_size(n_items, n_q, T, d, rk, rv, &need);
  if (rc) return rc;
  if (ws_bytes < need) {
    if (!caller_ws)
      return jolt_fail(JOLT_E_WORKSPACE, "jolt_attend_noalloc: the call needs %zu bytes of workspace, above the "
                       "fixed scratch of %zu bytes (split the items over several calls)", need, ws_bytes);
    return jolt_fail(JOLT_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  }
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  if (caller_ws) forget_spectra(ctx, ws, ws_bytes);
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ws);
  AttnItem *items; uint64_t *seeds; float *signs, *gk, *qr, *part;
  plan_attend(cv, n_items, n_q, T, d, rk, rv, &items, &seeds, &signs, &gk, &qr, &part);
  std::vector<AttnItem> hi(n_items);
  std::vector<uint64_t> hs(2 * (size_t)n_items);
  auto blob = [](const void *base, const BlobInfo &b) {
    const uint8_t *p8 = static_cast<const uint8_t *>(base);
    return AttnBlob{p8 + b.L.UT, p8 + b.L.Ud, p8 + b.L.G, reinterpret_cast<const int8_t *>(p8 + b.L.gexp),
                    p8 + b.L.codes, reinterpret_cast<const uint16_t *>(p8 + b.L.scales),
                    (int32_t)b.rT, (int32_t)b.rd, (int32_t)b.bits, (int32_t)b.f16};
  };
  for (int i = 0; i < n_items; ++i) {
    hi[i] = AttnItem{blob(k_blobs[i], kb[i]), blob(v_blobs[i], vb[i]), layers[i], 0};
    hs[2 * i] = kb[i].seed;
    hs[2 * i + 1] = vb[i].seed;
  }
  HIP_OK(hipMemcpyAsync(items, hi.data(), hi.size() * sizeof(AttnItem), hipMemcpyHostToDevice, st));
  HIP_OK(hipMemcpyAsync(seeds, hs.data(), hs.size() * sizeof(uint64_t), hipMemcpyHostToDevice, st));
  HIP_OK(launch_rotation_signs(seeds, 2 * n_items, d, signs, st));
  AttnArgs a{};
  a.items = items; a.signs = signs; a.Q = Q; a.O = O; a.gk = gk; a.qr = qr; a.part = part;
  a.n_items = n_items; a.n_q = n_q; a.heads = H; a.T = T; a.group = kb[0].group;
  a.chunks = (T + ATTN_CHUNK - 1) / ATTN_CHUNK; a.rk_max = std::max(rk, 1); a.rv_max = rv;
  a.scale = scale; a.inv_sqrt_d = (float)(1.0 / std::sqrt((double)d));
  StageTimer t(ctx, st, JOLT_STAGE_ATTEND);
  HIP_OK(launch_attend(a, d, st));
  return JOLT_OK;
}
}  // namespace

extern "C" int jolt_attend(jolt_ctx *ctx, int n_items, const void *const *k_blobs, const size_t *k_bytes,
                           const void *const *v_blobs, const size_t *v_bytes, const void *k_hdr_host,
                           const void *v_hdr_host, const int32_t *layers, int n_q, const float *Q,
                           float scale, float *O, void *ws, size_t ws_bytes, jolt_stream stream) {
  return attend_impl(ctx, n_items, k_blobs, k_bytes, v_blobs, v_bytes, k_hdr_host, v_hdr_host, layers, n_q,
                     Q, scale, O, ws, ws_bytes, true, stream);
}

extern "C" int jolt_attend_noalloc(jolt_ctx *ctx, int n_items, const void *const *k_blobs,
                                   const size_t *k_bytes, const void *const *v_blobs, const size_t *v_bytes,
                                   const void *k_hdr_host, const void *v_hdr_host, const int32_t *layers,
                                   int n_q, const float *Q, float scale, float *O, jolt_stream stream) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "jolt_attend_noalloc: ctx is null");
  if (!ctx->attend_scratch) return jolt_fail(JOLT_E_STATE, "jolt_attend_noalloc: no scratch for this context");
  return attend_impl(ctx, n_items, k_blobs, k_bytes, v_blobs, v_bytes, k_hdr_host, v_hdr_host, layers, n_q,
                     Q, scale, O, ctx->attend_scratch, ATTN_SCRATCH_BYTES, false, stream);
}

// ------------------------------------------------------------------------ debug export
extern "C" int jolt_debug_export(jolt_ctx *ctx, int what, int cell, void *dst, size_t dst_bytes,
                                 jolt_stream stream) {
  if (!ctx || !dst) return jolt_fail(JOLT_E_INVAL, "jolt_debug_export: null argument");
  const DebugState &g = ctx->dbg;
  if (!g.valid) return jolt_fail(JOLT_E_STATE, "jolt_debug_export: no compress call recorded");
  if (cell < 0 || cell >= g.n_cells) return jolt_fail(JOLT_E_INVAL, "cell out of range");
  hipStream_t st = (hipStream_t)stream;
  DeviceGuard dg;
  HIP_OK(dg.enter(ctx->device));
  if (what == 0 || what == 1) {
    const int rows = what == 0 ? g.T : g.d, cols = what == 0 ? g.rT[cell] : g.rd[cell];
    const float *src = what == 0 ? g.U + cell * g.u_stride : g.Ud + cell * g.ud_stride;
    const int64_t ld = what == 0 ? g.ldu : g.d;
    if (dst_bytes < (size_t)rows * cols * sizeof(float)) return jolt_fail(JOLT_E_WORKSPACE, "dst too small");
    if (cols == 0) return JOLT_OK;
    HIP_OK(hipMemcpy2DAsync(dst, cols * sizeof(float), src, ld * sizeof(float), cols * sizeof(float), rows,
                            hipMemcpyDeviceToDevice, st));
    return JOLT_OK;
  }
  if (what == 2) {
    const size_t n = (size_t)g.m * g.T * g.d * sizeof(float);
    if (dst_bytes < n) return jolt_fail(JOLT_E_WORKSPACE, "dst too small");
    if (reinterpret_cast<uintptr_t>(dst) & 15) return jolt_fail(JOLT_E_INVAL, "dst must be 16-byte aligned");
    // the recorded call's fused reconstruction, in its export mode, for this one cell
    FusedCell fc = g.fused[cell];
    fc.xt_out = static_cast<float *>(dst);
    HIP_OK(hipMemcpyAsync(g.fcell_dev + cell, &fc, sizeof fc, hipMemcpyHostToDevice, st));
    FusedArgs a = g.fargs;
    a.cells = g.fcell_dev + cell;
    a.signs = g.fargs.signs + (int64_t)cell * g.d;
    a.n_cells = 1;
    HIP_OK(launch_fused(a, FUSED_XTILDE, g.d, JOLT_F32, g.split, st));
    return JOLT_OK;
  }
  if (what == 3) {
    if (!g.Omega) return jolt_fail(JOLT_E_STATE, "no sketch in the recorded call");
    const size_t n = (size_t)g.N * g.ell * sizeof(uint16_t);
    if (dst_bytes < n) return jolt_fail(JOLT_E_WORKSPACE, "dst too small");
    HIP_OK(hipMemcpy2DAsync(dst, g.ell * sizeof(uint16_t), g.Omega + cell * g.om_stride,
                            g.ldo * sizeof(uint16_t), g.ell * sizeof(uint16_t), g.N,
                            hipMemcpyDeviceToDevice, st));
    return JOLT_OK;
  }
  return jolt_fail(JOLT_E_INVAL, "unknown export %d", what);
}

extern "C" int jolt_debug_set(jolt_ctx *ctx, int what, int64_t value) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: ctx is null");
  if (what == JOLT_DBG_INVIT_ITERS) {
    if (value < 0 || value > 8) return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: iterations must be in 0..8");
    ctx->invit_iters = (int)value;
    return JOLT_OK;
  }
  if (what == JOLT_DBG_TRD_LANES) {
    if (value < 1 || value > jolt_ctx::kTrdLanes)
      return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: tridiagonalisation lanes must be in 1..%d", jolt_ctx::kTrdLanes);
    ctx->trd_lanes_max = (int)value;
    return JOLT_OK;
  }
  if (what == JOLT_DBG_BULGE_SPIN) {
    if (value < 0 || value > SB_SPIN_DEFAULT)
      return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: bulge-chase wait bound must be in 0..%d", SB_SPIN_DEFAULT);
    ctx->bulge_spin = (int)value;
    return JOLT_OK;
  }
  if (what == JOLT_DBG_TRD_TWO_STAGE) {
    if (value < -1 || value > 1)
      return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: two-stage switch must be -1 (automatic), 0 or 1");
    ctx->trd_two_stage = (int)value;
    return JOLT_OK;
  }
  return jolt_fail(JOLT_E_INVAL, "jolt_debug_set: unknown setting %d", what);
}
