// C-ABI of the JoLT / FlashJoLT compression path: argument validation, workspace
// layout, orchestration of the gfx950 kernels, blob headers.  Every entry point
// validates its arguments before queuing device work and reports failures through
// a negative return code plus jolt_last_error().
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "../../include/jolt.h"
#include "host_util.h"
#include "kernels.h"
#include "jolt_internal.h"

// ------------------------------------------------------------------------ errors
static thread_local std::string g_err;

int jolt_fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int jolt_hip_fail(hipError_t e, const char *what, const char *file, int line) {
  return jolt_fail(JOLT_E_HIP, "HIP error %d (%s) in %s at %s:%d", (int)e, hipGetErrorString(e),
                   what, file, line);
}

extern "C" const char *jolt_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------------ context
extern "C" int jolt_create(jolt_ctx **ctx, int device) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "jolt_create: ctx is null");
  *ctx = nullptr;
  int ndev = 0;
  HIP_OK(hipGetDeviceCount(&ndev));
  if (device >= ndev) return jolt_fail(JOLT_E_INVAL, "jolt_create: device %d of %d", device, ndev);
  if (device < 0) HIP_OK(hipGetDevice(&device));
  // owned until every check has passed: no path leaks the context or reads it after release
  std::unique_ptr<jolt_ctx> c(new jolt_ctx());
  c->device = device;
  HIP_OK(hipGetDeviceProperties(&c->prop, device));
  const std::string arch(c->prop.gcnArchName);
  if (arch.find("gfx950") == std::string::npos)
    return jolt_fail(JOLT_E_UNSUPPORTED, "jolt_create: device arch %s is not gfx950", arch.c_str());
  {
    // set-up of the allocation-free entry point: this device's scratch address, once per device
    DeviceGuard dg;
    HIP_OK(dg.enter(device));
    HIP_OK(attend_scratch_address(device, &c->attend_scratch));
  }
  *ctx = c.release();
  return JOLT_OK;
}

extern "C" int jolt_destroy(jolt_ctx *ctx) {
  delete ctx;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ policies
extern "C" int jolt_q_cap(int T, double R) {
  if (T < 1 || !(R > 0.0)) return jolt_fail(JOLT_E_INVAL, "jolt_q_cap: T >= 1 and R > 0 required");
  const int qmin = R <= 4.0 ? 32 : 64;
  const int t32 = (T + 31) / 32;
  return std::min(std::max(qmin, t32), 512);
}

int validate_desc(const jolt_cell_desc *d) {
  if (!d) return jolt_fail(JOLT_E_INVAL, "cell descriptor is null");
  if (d->dtype != JOLT_F32 && d->dtype != JOLT_BF16)
    return jolt_fail(JOLT_E_INVAL, "dtype must be JOLT_F32 or JOLT_BF16");
  if (d->n_layers < 1 || d->n_heads < 1 || d->T < 1)
    return jolt_fail(JOLT_E_INVAL, "n_layers, n_heads and T must be >= 1");
  if (d->d != 32 && d->d != 64 && d->d != 128)
    return jolt_fail(JOLT_E_UNSUPPORTED, "d must be 32, 64 or 128 (got %d)", d->d);
  if (d->stride_token < d->d) return jolt_fail(JOLT_E_INVAL, "stride_token must be >= d");
  if ((d->stride_token % 8) || (d->stride_head % 8) || (d->stride_layer % 8))
    return jolt_fail(JOLT_E_INVAL, "strides must be multiples of 8 elements");
  if (d->stride_head < 0 || d->stride_layer < 0) return jolt_fail(JOLT_E_INVAL, "negative stride");
  const int64_t m = (int64_t)d->n_layers * d->n_heads;
  if (m * d->d > (1 << 26) || d->T > (1 << 20))
    return jolt_fail(JOLT_E_UNSUPPORTED, "cell too large (m*d <= 2^26, T <= 2^20)");
  return JOLT_OK;
}

int resolve_spectrum(const jolt_cell_desc *d, const jolt_spectrum_opts *o, SpecShape *sh) {
  int rc = validate_desc(d);
  if (rc) return rc;
  sh->m = d->n_layers * d->n_heads;
  sh->T = d->T;
  sh->d = d->d;
  sh->N = sh->m * d->d;
  sh->method = o ? o->method : JOLT_EXACT;
  const int r_cap = o ? o->r_max : 0;
  if (r_cap < 0) return jolt_fail(JOLT_E_INVAL, "r_max must be >= 0 (0 = no cap)");
  if (sh->method == JOLT_EXACT) {
    sh->n_lam_T = sh->T;
    sh->rT_max = std::min(sh->T, sh->N);
    if (r_cap > 0) sh->rT_max = std::min(sh->rT_max, r_cap);
    sh->q = sh->ell = 0;
    if (sh->T > 8192)
      return jolt_fail(JOLT_E_UNSUPPORTED, "exact token spectrum limited to T <= 8192 (use FlashJoLT)");
  } else if (sh->method == JOLT_FLASH) {
    if (o->oversample < 0 || o->power_iters < 0 || o->power_iters > 16)
      return jolt_fail(JOLT_E_INVAL, "oversample >= 0 and 0 <= power_iters <= 16 required");
    int q = o->q;
    if (q == 0) {
      q = jolt_q_cap(sh->T, o->ratio);
      if (q < 0) return q;
    }
    if (q < 1) return jolt_fail(JOLT_E_INVAL, "q must be >= 1");
    sh->ell = std::min<int64_t>(std::min<int64_t>((int64_t)q + o->oversample, sh->T), sh->N);
    sh->q = std::min(q, sh->ell);
    sh->n_lam_T = sh->q + 1;
    sh->rT_max = r_cap > 0 ? std::min(sh->q, r_cap) : sh->q;
    if (sh->ell > 1024) return jolt_fail(JOLT_E_UNSUPPORTED, "sketch width l must be <= 1024");
  } else {
    return jolt_fail(JOLT_E_INVAL, "method must be JOLT_EXACT or JOLT_FLASH");
  }
  return JOLT_OK;
}

extern "C" int jolt_spectrum_len(const jolt_cell_desc *desc, const jolt_spectrum_opts *opts,
                                 int32_t *n_lam_T, int32_t *rT_max) {
  SpecShape sh;
  int rc = resolve_spectrum(desc, opts, &sh);
  if (rc) return rc;
  if (n_lam_T) *n_lam_T = sh.n_lam_T;
  if (rT_max) *rT_max = sh.rT_max;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ blob format
BlobLayout blob_layout(int64_t m, int64_t T, int64_t d, int64_t rT, int64_t rd, int64_t bits,
                       int64_t group, int64_t fb) {
  auto al = [](int64_t x) { return (x + 255) / 256 * 256; };
  BlobLayout L;
  int64_t pos = al(kHeaderBytes);
  L.UT = pos; pos = al(pos + T * rT * fb);
  L.Ud = pos; pos = al(pos + d * rd * fb);
  L.G = pos; pos = al(pos + m * rT * rd * fb);
  L.gexp = pos; pos = al(pos + m);
  L.scales = pos; pos = al(pos + (bits ? 2 * (m * T * d / group) : 0));
  L.codes = pos; pos = pos + (m * T * d * bits) / 8;
  L.total = pos;
  return L;
}

int validate_params(const jolt_cell_desc *d, const jolt_params *p, int rT_max) {
  if (!p) return jolt_fail(JOLT_E_INVAL, "params is null");
  if (p->bits != 0 && p->bits != 2 && p->bits != 4 && p->bits != 8)
    return jolt_fail(JOLT_E_INVAL, "bits must be 0, 2, 4 or 8 (got %d)", p->bits);
  if (p->group < 8 || p->group > d->d || (d->d % p->group) || (p->group % 8))
    return jolt_fail(JOLT_E_INVAL, "group must divide d and be a multiple of 8 (got %d)", p->group);
  if (p->r_T < 0 || p->r_d < 0 || (p->r_T == 0) != (p->r_d == 0))
    return jolt_fail(JOLT_E_INVAL, "ranks must be >= 0 with r_T = 0 iff r_d = 0");
  if (p->r_T > rT_max) return jolt_fail(JOLT_E_INVAL, "r_T = %d exceeds %d", p->r_T, rT_max);
  if (p->r_d > d->d) return jolt_fail(JOLT_E_INVAL, "r_d = %d exceeds d = %d", p->r_d, d->d);
  if (p->factor_dtype != JOLT_FACTOR_F16 && p->factor_dtype != JOLT_FACTOR_F32)
    return jolt_fail(JOLT_E_INVAL, "factor_dtype must be JOLT_FACTOR_F16 or JOLT_FACTOR_F32");
  return JOLT_OK;
}

extern "C" int jolt_compressed_size(const jolt_cell_desc *desc, const jolt_params *p, size_t *bytes) {
  int rc = validate_desc(desc);
  if (rc) return rc;
  const int m = desc->n_layers * desc->n_heads;
  rc = validate_params(desc, p, std::min(desc->T, m * desc->d));
  if (rc) return rc;
  if (!bytes) return jolt_fail(JOLT_E_INVAL, "bytes is null");
  const int fb = p->factor_dtype == JOLT_FACTOR_F16 ? 2 : 4;
  *bytes = (size_t)blob_layout(m, desc->T, desc->d, p->r_T, p->r_d, p->bits, p->group, fb).total;
  return JOLT_OK;
}

void fill_header(uint8_t *h, const jolt_cell_desc *d, const jolt_params *p, int method) {
  const int m = d->n_layers * d->n_heads;
  const int fb = p->factor_dtype == JOLT_FACTOR_F16 ? 2 : 4;
  BlobLayout L = blob_layout(m, d->T, d->d, p->r_T, p->r_d, p->bits, p->group, fb);
  std::memset(h, 0, kHeaderBytes);
  std::memcpy(h, "JOLT", 4);
  uint32_t u[11] = {1u, (uint32_t)(d->dtype == JOLT_BF16 ? 1 : 0),
                    (uint32_t)(p->factor_dtype == JOLT_FACTOR_F16 ? 1 : 0), (uint32_t)m,
                    (uint32_t)d->T, (uint32_t)d->d, (uint32_t)p->r_T, (uint32_t)p->r_d,
                    (uint32_t)p->bits, (uint32_t)p->group, (uint32_t)method};
  std::memcpy(h + 4, u, sizeof u);
  std::memcpy(h + 48, &p->seed, 8);
  uint64_t o[7] = {(uint64_t)L.UT, (uint64_t)L.Ud, (uint64_t)L.G, (uint64_t)L.gexp,
                   (uint64_t)L.scales, (uint64_t)L.codes, (uint64_t)L.total};
  std::memcpy(h + 56, o, sizeof o);
  uint32_t heads = (uint32_t)d->n_heads;
  std::memcpy(h + 112, &heads, 4);
}

int parse_header(const uint8_t *h, size_t blob_bytes, BlobInfo *bi) {
  if (std::memcmp(h, "JOLT", 4) != 0) return jolt_fail(JOLT_E_BLOB, "blob magic mismatch");
  uint32_t u[11];
  std::memcpy(u, h + 4, sizeof u);
  if (u[0] != 1) return jolt_fail(JOLT_E_BLOB, "unsupported blob version %u", u[0]);
  bi->in_bf16 = u[1]; bi->f16 = u[2]; bi->m = u[3]; bi->T = u[4]; bi->d = u[5];
  bi->rT = u[6]; bi->rd = u[7]; bi->bits = u[8]; bi->group = u[9]; bi->method = u[10];
  std::memcpy(&bi->seed, h + 48, 8);
  uint64_t o[7];
  std::memcpy(o, h + 56, sizeof o);
  std::memcpy(&bi->heads, h + 112, 4);
  BlobLayout L = blob_layout(bi->m, bi->T, bi->d, bi->rT, bi->rd, bi->bits, bi->group ? bi->group : 1,
                             bi->f16 ? 2 : 4);
  if (bi->group == 0 || (bi->bits != 0 && bi->bits != 2 && bi->bits != 4 && bi->bits != 8) ||
      (uint64_t)L.UT != o[0] || (uint64_t)L.Ud != o[1] || (uint64_t)L.G != o[2] ||
      (uint64_t)L.gexp != o[3] || (uint64_t)L.scales != o[4] || (uint64_t)L.codes != o[5] ||
      (uint64_t)L.total != o[6])
    return jolt_fail(JOLT_E_BLOB, "blob header section table is inconsistent");
  if ((size_t)L.total > blob_bytes) return jolt_fail(JOLT_E_BLOB, "blob shorter than its header says");
  bi->L = L;
  return JOLT_OK;
}

// ------------------------------------------------------------------------ profiling
constexpr size_t kProfPendingMax = 4096;
static int prof_drain(jolt_ctx *c);

static hipEvent_t pool_get(jolt_ctx *c) {
  if (!c->prof_pool.empty()) {
    hipEvent_t e = c->prof_pool.back();
    c->prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

StageTimer::StageTimer(jolt_ctx *c, hipStream_t s, int stage_) : ctx(c), st(s), stage(stage_) {
  if (!ctx || !ctx->prof_on) return;
  a = pool_get(ctx);
  if (a && hipEventRecord(a, st) != hipSuccess) {
    ctx->prof_pool.push_back(a);
    a = nullptr;
  }
}

StageTimer::~StageTimer() {
  if (!a) return;
  hipEvent_t b = pool_get(ctx);
  if (b && hipEventRecord(b, st) == hipSuccess) {
    ctx->prof_pending.push_back(ProfRecord{stage, a, b});
    // bounded number of outstanding events: read the pending intervals (a host wait)
    if (ctx->prof_pending.size() >= kProfPendingMax) (void)prof_drain(ctx);
  } else {
    ctx->prof_pool.push_back(a);
    if (b) ctx->prof_pool.push_back(b);
  }
}

jolt_ctx::~jolt_ctx() {
  for (int g = 0; g < kTrdLanes; ++g) {
    if (trd_exec[g]) (void)hipGraphExecDestroy(trd_exec[g]);
    if (cap_stream[g]) (void)hipStreamDestroy(cap_stream[g]);
    if (trd_join[g]) (void)hipEventDestroy(trd_join[g]);
  }
  if (trd_fork) (void)hipEventDestroy(trd_fork);
  for (auto &r : prof_pending) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
  for (auto e : prof_pool) (void)hipEventDestroy(e);
}

static int prof_drain(jolt_ctx *c) {
  for (auto &r : c->prof_pending) {
    HIP_OK(hipEventSynchronize(r.b));
    float ms = 0.f;
    HIP_OK(hipEventElapsedTime(&ms, r.a, r.b));
    c->prof_ms[r.stage] += ms;
    c->prof_n[r.stage] += 1;
    c->prof_pool.push_back(r.a);
    c->prof_pool.push_back(r.b);
  }
  c->prof_pending.clear();
  return JOLT_OK;
}

extern "C" int jolt_profile_enable(jolt_ctx *ctx, int on) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "ctx is null");
  ctx->prof_on = on != 0;
  return JOLT_OK;
}

extern "C" int jolt_profile_reset(jolt_ctx *ctx) {
  if (!ctx) return jolt_fail(JOLT_E_INVAL, "ctx is null");
  int rc = prof_drain(ctx);
  if (rc) return rc;
  for (int i = 0; i < JOLT_STAGE_COUNT; ++i) { ctx->prof_ms[i] = 0.0; ctx->prof_n[i] = 0; }
  return JOLT_OK;
}

extern "C" int jolt_profile_read(jolt_ctx *ctx, int stage, double *total_ms, int64_t *launches) {
  if (!ctx || stage < 0 || stage >= JOLT_STAGE_COUNT) return jolt_fail(JOLT_E_INVAL, "bad profile query");
  int rc = prof_drain(ctx);
  if (rc) return rc;
  if (total_ms) *total_ms = ctx->prof_ms[stage];
  if (launches) *launches = ctx->prof_n[stage];
  return JOLT_OK;
}
