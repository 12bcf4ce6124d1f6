// Internal host-side declarations of the C-ABI implementation.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "../../include/jolt.h"
#include "kernels.h"

constexpr int kHeaderBytes = 128;

struct SpecShape {
  int m = 0, T = 0, d = 0, N = 0, method = 0;
  int n_lam_T = 0, rT_max = 0, q = 0, ell = 0;
};

struct BlobLayout {
  int64_t UT = 0, Ud = 0, G = 0, gexp = 0, scales = 0, codes = 0, total = 0;
};

struct BlobInfo {
  uint32_t in_bf16, f16, m, T, d, rT, rd, bits, group, method, heads;
  uint64_t seed;
  BlobLayout L;
};

// State a jolt_compress call may reuse from the preceding jolt_spectrum call.
// batch work (matrices x order) from which the automatic choice takes the two-stage reduction
constexpr int64_t kTwoStageMinWork = 32 * 4096;

struct SpecKey {
  bool valid = false;
  const void *ws = nullptr;
  size_t ws_bytes = 0;
  jolt_cell_desc desc{};
  jolt_spectrum_opts opts{};
  std::vector<const void *> X;
  std::vector<uint64_t> seeds;
  int32_t token_refl_off = 0;   // reduction that left the token reflectors (1 one-stage, else the band)
};

// Forget every recorded spectrum whose workspace overlaps [ws, ws + bytes), except `keep`.
void forget_spectra(jolt_ctx *ctx, const void *ws, size_t bytes, const SpecKey *keep = nullptr);

struct DebugState {
  bool valid = false;
  int n_cells = 0, T = 0, d = 0, m = 0, N = 0, ell = 0;
  std::vector<int> rT, rd;
  const float *U = nullptr, *Ud = nullptr;
  const uint16_t *Omega = nullptr;
  int64_t u_stride = 0, ldu = 0, ud_stride = 0, om_stride = 0, ldo = 0;
  // the fused reconstruction of the call (its records, device table and arguments)
  std::vector<FusedCell> fused;
  FusedCell *fcell_dev = nullptr;
  FusedArgs fargs{};
  bool split = false;
};

struct ProfRecord {
  int stage;
  hipEvent_t a, b;
};

struct jolt_ctx {
  int device = 0;
  hipDeviceProp_t prop{};
  // spectra left in caller workspaces by jolt_spectrum / jolt_compress, one per workspace
  std::vector<SpecKey> specs;
  DebugState dbg;
  std::vector<GemmProblem> tab_host;
  bool prof_on = false;
  std::vector<ProfRecord> prof_pending;
  std::vector<hipEvent_t> prof_pool;
  double prof_ms[JOLT_STAGE_COUNT] = {};
  int64_t prof_n[JOLT_STAGE_COUNT] = {};
  // replay of the fixed launch sequence of the blocked tridiagonalisation: the batch is
  // split into up to kTrdLanes groups of matrices, each captured once and replayed on a
  // stream of its own (the first on the call's stream: with the private streams, four in
  // all, the hardware queues of a process), so that one group's latency-bound column
  // kernels run beside another group's bandwidth-bound mat-vec (default stream priority)
  static constexpr int kTrdLanes = 4;
  hipStream_t cap_stream[kTrdLanes] = {};
  hipGraphExec_t trd_exec[kTrdLanes] = {};
  hipEvent_t trd_fork = nullptr, trd_join[kTrdLanes] = {};
  int trd_lanes = 0;               // lanes of the captured graphs
  int trd_lanes_max = kTrdLanes;   // JOLT_DBG_TRD_LANES
  std::vector<const void *> trd_key;
  int trd_two_stage = -1;          // JOLT_DBG_TRD_TWO_STAGE: 1 two-stage, 0 one-stage, -1 by batch size
  int bulge_spin = SB_SPIN_DEFAULT; // JOLT_DBG_BULGE_SPIN: bound of the bulge chase's waits
  int invit_iters = 2;            // inverse-iteration sweeps (test hook jolt_debug_set)
  void *attend_scratch = nullptr; // this device's fixed attention scratch (device address)
  ~jolt_ctx();
};

// Brackets device work queued on `st` while alive (no-op unless profiling is enabled).
struct StageTimer {
  jolt_ctx *ctx;
  hipStream_t st;
  int stage;
  hipEvent_t a = nullptr;
  StageTimer(jolt_ctx *c, hipStream_t s, int stage_);
  ~StageTimer();
};

int validate_desc(const jolt_cell_desc *d);
int resolve_spectrum(const jolt_cell_desc *d, const jolt_spectrum_opts *o, SpecShape *sh);
int validate_params(const jolt_cell_desc *d, const jolt_params *p, int rT_max);
BlobLayout blob_layout(int64_t m, int64_t T, int64_t d, int64_t rT, int64_t rd, int64_t bits,
                       int64_t group, int64_t fb);
void fill_header(uint8_t *h, const jolt_cell_desc *d, const jolt_params *p, int method);
int parse_header(const uint8_t *h, size_t blob_bytes, BlobInfo *bi);
