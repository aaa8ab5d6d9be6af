// C ABI of the library: argument validation, handle management and status
// reporting around the factorisation and sweep launches.
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace g2d {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

gptq2d_status hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return e == hipErrorOutOfMemory ? GPTQ2D_ERR_OOM : GPTQ2D_ERR_HIP;
}

static gptq2d_status fail(gptq2d_status s, const std::string& msg) {
  set_error(msg);
  return s;
}

static int round_up(int v, int a) { return (v + a - 1) / a * a; }

static void free_all(Factors* f) {
  for (void* p : f->allocations) (void)hipFree(p);
  f->allocations.clear();
  if (f->ev_near) (void)hipEventDestroy(f->ev_near);
  if (f->ev_far) (void)hipEventDestroy(f->ev_far);
  if (f->ev_far1) (void)hipEventDestroy(f->ev_far1);
  for (hipEvent_t ev : f->stage_ev) (void)hipEventDestroy(ev);
  f->stage_ev.clear();
  if (f->aux) (void)hipStreamDestroy(f->aux);
  if (f->ev_own) (void)hipEventDestroy(f->ev_own);
  if (f->own) (void)hipStreamDestroy(f->own);
  f->ev_near = f->ev_far = f->ev_far1 = f->ev_own = nullptr;
  f->aux = f->own = nullptr;
  free_schedule(f->sched);
}

static gptq2d_status alloc(Factors* f, void** p, size_t bytes) {
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) return hip_fail(e, "device allocation");
  f->allocations.push_back(*p);
  return GPTQ2D_OK;
}

static int env_int(const char* name, int def) {
  const char* v = getenv(name);
  if (!v || !*v) return def;
  return atoi(v);
}

gptq2d_status check_device(const Factors* f) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != f->device)
    return fail(GPTQ2D_ERR_INVALID_ARG, "the current device is not the device of the handle");
  return GPTQ2D_OK;
}

gptq2d_status check_round_args(const Factors* f, gptq2d_dtype dt, const void* X, int64_t ldx,
                               const int32_t* Z, int64_t ldz, const void* Y, int64_t ldy) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  if (dt != GPTQ2D_F32 && dt != GPTQ2D_F64) return fail(GPTQ2D_ERR_INVALID_ARG, "bad dtype");
  if (!X || !Z) return fail(GPTQ2D_ERR_INVALID_ARG, "X or Z is NULL");
  if (ldx < f->n || ldz < f->n || (Y && ldy < f->n))
    return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
  return GPTQ2D_OK;
}

}  // namespace g2d

using namespace g2d;

// The error word at the head of a round workspace (single or batched), after
// the stream has been synchronised, as a status.
static gptq2d_status round_flags_status(const void* workspace) {
  int flags = 0;
  hipError_t e = hipMemcpy(&flags, workspace, sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
  if (flags & FLAG_NONFINITE) return fail(GPTQ2D_ERR_NONFINITE, "X held a NaN or an infinity");
  if (flags & FLAG_OVERFLOW) return fail(GPTQ2D_ERR_OVERFLOW, "a rounded value does not fit in int32");
  if (flags & FLAG_TIMEOUT) return fail(GPTQ2D_ERR_TIMEOUT, "a wave waited too long for its neighbour");
  return GPTQ2D_OK;
}

extern "C" {

gptq2d_status gptq2d_factors_create(int m, int n, gptq2d_factors_t* out) {
  if (!out) return fail(GPTQ2D_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (m < 1 || n < 1 || m > 65536 || n > 65536)
    return fail(GPTQ2D_ERR_INVALID_ARG, "m and n must lie in [1, 65536]");
  gptq2d_factors_s* f = new gptq2d_factors_s();
  f->m = m;
  f->n = n;
  f->mp = round_up(m, TB);
  f->np = round_up(n, TB);
  f->MT = f->mp / TB;
  f->NT = f->np / TB;
  hipError_t he = hipGetDevice(&f->device);
  if (he != hipSuccess) {
    delete f;
    return hip_fail(he, "hipGetDevice");
  }
  const size_t mp = (size_t)f->mp, np = (size_t)f->np;
  gptq2d_status st = GPTQ2D_OK;
  void* p = nullptr;
  auto A = [&](double** dst, size_t count) {
    if (st != GPTQ2D_OK) return;
    st = alloc(f, &p, count * sizeof(double));
    if (st == GPTQ2D_OK) *dst = (double*)p;
  };
  A(&f->L, mp * mp);
  A(&f->U, np * np);
  A(&f->dL, mp);
  A(&f->dU, np);
  A(&f->gram[0], mp * mp);
  A(&f->inv[0], mp * mp);
  A(&f->dinv[0], mp * TB);
  A(&f->gram[1], np * np);
  A(&f->inv[1], np * np);
  A(&f->dinv[1], np * TB);
  if (hipDeviceGetAttribute(&f->cus, hipDeviceAttributeMultiprocessorCount, f->device) != hipSuccess ||
      f->cus <= 0)
    f->cus = 256;
  const size_t gpd = gram_part_doubles(f->m, f->n, f->cus);
  if (gpd > 0) A(&f->gpart, gpd);
  const size_t gev = gram_env_ints(f->m, f->n);
  if (gev > 0 && st == GPTQ2D_OK) {
    st = alloc(f, &p, gev * sizeof(int));
    if (st == GPTQ2D_OK) f->genv = (int*)p;
  }
  if (st == GPTQ2D_OK) {
    st = alloc(f, &p, 256);
    if (st == GPTQ2D_OK) {
      f->flags = (int*)p;
      st = alloc(f, &f->d_fac, fac_static_bytes());
    }
    if (st == GPTQ2D_OK) st = upload_fac_static(*f);
    if (st == GPTQ2D_OK) {
      he = hipMemset(f->flags, 0, 256);
      if (he != hipSuccess) st = hip_fail(he, "hipMemset");
    }
  }
  if (st == GPTQ2D_OK) {
    he = hipStreamCreateWithFlags(&f->aux, hipStreamNonBlocking);
    if (he == hipSuccess) he = hipEventCreateWithFlags(&f->ev_near, hipEventDisableTiming);
    if (he == hipSuccess) he = hipEventCreateWithFlags(&f->ev_far, hipEventDisableTiming);
    if (he == hipSuccess) he = hipEventCreateWithFlags(&f->ev_far1, hipEventDisableTiming);
    if (he != hipSuccess) st = hip_fail(he, "stream / event creation");
  }
  if (st == GPTQ2D_OK) {
    // far-delivery batch width in source tiles: wider batches mean fewer
    // read-modify-writes of the feedback buffers but coarser products; five
    // measured best from about 128 tiles per side on, four below
    const int g = std::max(f->MT, f->NT) > 64 ? 5 : 4;
    st = build_schedule(*f, env_int("GPTQ2D_BATCH", g));
  }
  if (st != GPTQ2D_OK) {
    free_all(f);
    delete f;
    return st;
  }
  *out = f;
  return GPTQ2D_OK;
}

void gptq2d_factors_destroy(gptq2d_factors_t f) {
  if (!f) return;
  free_all(f);
  delete f;
}

gptq2d_status gptq2d_factors_shape(gptq2d_factors_t f, int* m, int* n) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  if (m) *m = f->m;
  if (n) *n = f->n;
  return GPTQ2D_OK;
}

gptq2d_status gptq2d_factors_set_order(gptq2d_factors_t f, int reverse) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  f->rev = reverse ? 1 : 0;
  return GPTQ2D_OK;
}

gptq2d_status gptq2d_factor_compute(gptq2d_factors_t f, gptq2d_dtype dt, const void* A,
                                    int64_t lda, const void* B, int64_t ldb, void* stream) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  if (dt != GPTQ2D_F32 && dt != GPTQ2D_F64) return fail(GPTQ2D_ERR_INVALID_ARG, "bad dtype");
  if (!A || !B) return fail(GPTQ2D_ERR_INVALID_ARG, "A or B is NULL");
  if (lda < f->m || ldb < f->n) return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
  gptq2d_status st = check_device(f);
  if (st != GPTQ2D_OK) return st;
  return launch_factor(*f, dt, A, lda, B, ldb, (hipStream_t)stream);
}

gptq2d_status gptq2d_factor_check(gptq2d_factors_t f, void* stream) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  int flags = 0;
  e = hipMemcpy(&flags, f->flags, sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
  if (flags & FLAG_SINGULAR)
    return fail(GPTQ2D_ERR_SINGULAR, "a Gram pivot was not positive and finite (A or B singular)");
  return GPTQ2D_OK;
}

size_t gptq2d_factor_batched_workspace_size(int count) {
  return count < 1 ? 0 : (factor_batch_table_bytes(count) + 255) / 256 * 256;
}

gptq2d_status gptq2d_factor_batched(int count, const gptq2d_factors_t* f, gptq2d_dtype dt,
                                    const void* const* A, const int64_t* lda, const void* const* B,
                                    const int64_t* ldb, void* workspace, size_t ws_bytes,
                                    void* stream) {
  if (count < 1) return fail(GPTQ2D_ERR_INVALID_ARG, "count must be at least 1");
  if (!f || !A || !lda || !B || !ldb) return fail(GPTQ2D_ERR_INVALID_ARG, "an argument array is NULL");
  if (dt != GPTQ2D_F32 && dt != GPTQ2D_F64) return fail(GPTQ2D_ERR_INVALID_ARG, "bad dtype");
  for (int p = 0; p < count; ++p) {
    if (!f[p]) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
    if (!A[p] || !B[p]) return fail(GPTQ2D_ERR_INVALID_ARG, "A or B is NULL");
    if (lda[p] < f[p]->m || ldb[p] < f[p]->n)
      return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
    for (int q = 0; q < p; ++q)
      if (f[q] == f[p]) return fail(GPTQ2D_ERR_INVALID_ARG, "a handle appears twice");
    gptq2d_status st = check_device(f[p]);
    if (st != GPTQ2D_OK) return st;
  }
  if (!workspace || ws_bytes < gptq2d_factor_batched_workspace_size(count))
    return fail(GPTQ2D_ERR_WORKSPACE,
                "workspace missing or smaller than gptq2d_factor_batched_workspace_size()");
  if (((uintptr_t)workspace) % 256 != 0)
    return fail(GPTQ2D_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  // groups of problems of one shape (in order of first appearance), each
  // factorised in common launches, the groups side by side
  std::vector<int> order;
  std::vector<std::pair<int, int>> groups;  // (first position in order, size)
  std::vector<char> taken(count, 0);
  for (int p = 0; p < count; ++p) {
    if (taken[p]) continue;
    const int first = (int)order.size();
    for (int q = p; q < count; ++q)
      if (!taken[q] && f[q]->m == f[p]->m && f[q]->n == f[p]->n) {
        taken[q] = 1;
        order.push_back(q);
      }
    groups.emplace_back(first, (int)order.size() - first);
  }
  std::vector<Factors*> gf(count);
  std::vector<const void*> gA(count), gB(count);
  std::vector<int64_t> glda(count), gldb(count);
  for (int i = 0; i < count; ++i) {
    gf[i] = f[order[i]];
    gA[i] = A[order[i]];
    gB[i] = B[order[i]];
    glda[i] = lda[order[i]];
    gldb[i] = ldb[order[i]];
  }
  for (const auto& g : groups) {
    Factors* h = gf[g.first];
    if (!h->own) {
      hipError_t e = hipStreamCreateWithFlags(&h->own, hipStreamNonBlocking);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&h->ev_own, hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail(e, "stream / event creation");
    }
  }
  hipStream_t s = (hipStream_t)stream;
  hipEvent_t start = nullptr;
  hipError_t e = hipEventCreateWithFlags(&start, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(start, s);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  gptq2d_status st = GPTQ2D_OK;
  for (const auto& g : groups) {
    const int i0 = g.first, cnt = g.second;
    Factors* h = gf[i0];
    e = hipStreamWaitEvent(h->own, start, 0);
    if (e != hipSuccess) {
      st = hip_fail(e, "hipStreamWaitEvent");
      break;
    }
    if (cnt == 1)
      st = launch_factor(*h, dt, gA[i0], glda[i0], gB[i0], gldb[i0], h->own);
    else
      st = launch_factor_batched(cnt, &gf[i0], dt, &gA[i0], &glda[i0], &gB[i0], &gldb[i0],
                                 (char*)workspace + factor_batch_table_bytes(i0), h->own);
    if (st != GPTQ2D_OK) break;
    e = hipEventRecord(h->ev_own, h->own);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, h->ev_own, 0);
    if (e != hipSuccess) {
      st = hip_fail(e, "hipEventRecord");
      break;
    }
  }
  (void)hipEventDestroy(start);  // released once the recorded work is done
  return st;
}

gptq2d_status gptq2d_factor_batched_check(int count, const gptq2d_factors_t* f, void* stream) {
  if (count < 1 || !f) return fail(GPTQ2D_ERR_INVALID_ARG, "empty batch");
  for (int p = 0; p < count; ++p) {
    gptq2d_status st = gptq2d_factor_check(f[p], stream);
    if (st != GPTQ2D_OK) return st;
  }
  return GPTQ2D_OK;
}

gptq2d_status gptq2d_factor(int m, int n, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, void* stream, gptq2d_factors_t* out) {
  if (!out) return fail(GPTQ2D_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  gptq2d_factors_t f = nullptr;
  gptq2d_status st = gptq2d_factors_create(m, n, &f);
  if (st != GPTQ2D_OK) return st;
  st = gptq2d_factor_compute(f, dt, A, lda, B, ldb, stream);
  if (st == GPTQ2D_OK) st = gptq2d_factor_check(f, stream);
  if (st != GPTQ2D_OK) {
    gptq2d_factors_destroy(f);
    return st;
  }
  *out = f;
  return GPTQ2D_OK;
}

gptq2d_status gptq2d_factors_export(gptq2d_factors_t f, double* L, int64_t ldl, double* U,
                                    int64_t ldu, double* lamL, double* lamU, void* stream) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  if ((L && ldl < f->m) || (U && ldu < f->n))
    return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
  gptq2d_status st = check_device(f);
  if (st != GPTQ2D_OK) return st;
  return launch_export(*f, L, ldl, U, ldu, lamL, lamU, (hipStream_t)stream);
}

gptq2d_status gptq2d_factors_import(gptq2d_factors_t f, const double* L, int64_t ldl,
                                    const double* U, int64_t ldu, const double* lamL,
                                    const double* lamU, void* stream) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  if (!L || !U || !lamL || !lamU) return fail(GPTQ2D_ERR_INVALID_ARG, "a factor pointer is NULL");
  if (ldl < f->m || ldu < f->n) return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
  gptq2d_status st = check_device(f);
  if (st != GPTQ2D_OK) return st;
  return launch_import(*f, L, ldl, U, ldu, lamL, lamU, (hipStream_t)stream);
}

size_t gptq2d_round_workspace_size(gptq2d_factors_t f) { return f ? workspace_bytes(*f) : 0; }

gptq2d_status gptq2d_round(gptq2d_factors_t f, gptq2d_dtype dt, const void* X, int64_t ldx,
                           int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                           void* workspace, size_t ws_bytes, void* stream) {
  const gptq2d_status sa = check_round_args(f, dt, X, ldx, Z, ldz, Y, ldy);
  if (sa != GPTQ2D_OK) return sa;
  if (!workspace || ws_bytes < workspace_bytes(*f))
    return fail(GPTQ2D_ERR_WORKSPACE, "workspace missing or smaller than gptq2d_round_workspace_size()");
  if (((uintptr_t)workspace) % 256 != 0)
    return fail(GPTQ2D_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  gptq2d_status st = check_device(f);
  if (st != GPTQ2D_OK) return st;
  Workspace ws = workspace_carve(*f, workspace);
  return launch_round(*f, dt, X, ldx, Z, ldz, Y, ldy, objective, ws, (hipStream_t)stream);
}

gptq2d_status gptq2d_round_check(gptq2d_factors_t f, const void* workspace, void* stream) {
  if (!f || !workspace) return fail(GPTQ2D_ERR_INVALID_ARG, "handle or workspace is NULL");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  return round_flags_status(workspace);
}

size_t gptq2d_round_batched_workspace_size(int count, const gptq2d_factors_t* f) {
  if (count < 1 || !f) return 0;
  for (int p = 0; p < count; ++p)
    if (!f[p]) return 0;
  return batched_workspace_bytes(count, (const Factors* const*)f);
}

gptq2d_status gptq2d_round_batched(int count, const gptq2d_factors_t* f, gptq2d_dtype dt,
                                   const void* const* X, const int64_t* ldx, int32_t* const* Z,
                                   const int64_t* ldz, void* const* Y, const int64_t* ldy,
                                   double* objective, void* workspace, size_t ws_bytes,
                                   void* stream) {
  if (count < 1) return fail(GPTQ2D_ERR_INVALID_ARG, "count must be at least 1");
  if (!f || !X || !ldx || !Z || !ldz) return fail(GPTQ2D_ERR_INVALID_ARG, "an argument array is NULL");
  if ((Y == nullptr) != (ldy == nullptr)) return fail(GPTQ2D_ERR_INVALID_ARG, "Y and ldy must both be given or both NULL");
  if (dt != GPTQ2D_F32 && dt != GPTQ2D_F64) return fail(GPTQ2D_ERR_INVALID_ARG, "bad dtype");
  for (int p = 0; p < count; ++p) {
    if (!f[p]) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
    if (!X[p] || !Z[p]) return fail(GPTQ2D_ERR_INVALID_ARG, "X or Z is NULL");
    if (ldx[p] < f[p]->n || ldz[p] < f[p]->n || (Y && Y[p] && ldy[p] < f[p]->n))
      return fail(GPTQ2D_ERR_INVALID_ARG, "leading dimension too small");
    gptq2d_status st = check_device(f[p]);
    if (st != GPTQ2D_OK) return st;
  }
  const Factors* const* fs = (const Factors* const*)f;
  if (!workspace || ws_bytes < batched_workspace_bytes(count, fs))
    return fail(GPTQ2D_ERR_WORKSPACE,
                "workspace missing or smaller than gptq2d_round_batched_workspace_size()");
  if (((uintptr_t)workspace) % 256 != 0)
    return fail(GPTQ2D_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return launch_round_batched(count, fs, dt, X, ldx, Z, ldz, Y, ldy, objective, workspace,
                              (hipStream_t)stream);
}

gptq2d_status gptq2d_round_batched_check(const void* workspace, void* stream) {
  if (!workspace) return fail(GPTQ2D_ERR_INVALID_ARG, "workspace is NULL");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  return round_flags_status(workspace);
}

gptq2d_status gptq2d_stage_timing(gptq2d_factors_t f, int enable) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  f->stage_timing = enable != 0;
  f->stage_ev_used = 0;
  return GPTQ2D_OK;
}

gptq2d_status gptq2d_stage_time(gptq2d_factors_t f, double* total_ms, int64_t* launches) {
  if (!f) return fail(GPTQ2D_ERR_INVALID_ARG, "handle is NULL");
  double sum = 0.0;
  const size_t used = f->stage_ev_used;
  if (used) {
    hipError_t e = hipEventSynchronize(f->stage_ev[used - 1]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  }
  for (size_t i = 0; i + 1 < used; i += 2) {
    float ms = 0.0f;
    hipError_t e = hipEventElapsedTime(&ms, f->stage_ev[i], f->stage_ev[i + 1]);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    sum += ms;
  }
  if (total_ms) *total_ms = sum;
  if (launches) *launches = (int64_t)(used / 2);
  f->stage_ev_used = 0;
  return GPTQ2D_OK;
}

const char* gptq2d_status_string(gptq2d_status s) {
  switch (s) {
    case GPTQ2D_OK: return "ok";
    case GPTQ2D_ERR_INVALID_ARG: return "invalid argument";
    case GPTQ2D_ERR_SINGULAR: return "singular basis";
    case GPTQ2D_ERR_NONFINITE: return "non-finite input";
    case GPTQ2D_ERR_OOM: return "out of device memory";
    case GPTQ2D_ERR_HIP: return "HIP runtime error";
    case GPTQ2D_ERR_WORKSPACE: return "workspace missing or too small";
    case GPTQ2D_ERR_OVERFLOW: return "rounded value outside int32";
    case GPTQ2D_ERR_TIMEOUT: return "internal wait timed out";
  }
  return "unknown status";
}

const char* gptq2d_last_error(void) { return g_last_error.c_str(); }

int gptq2d_version(void) { return 100; }

int64_t gptq2d_schedule_tasks(int m, int n, int g, int32_t* tasks, int64_t cap, int32_t* offsets) {
  if (m < 1 || n < 1 || m > 65536 || n > 65536 || g < 1) {
    set_error("bad shape or batch width");
    return -1;
  }
  const int MT = (m + TB - 1) / TB, NTt = (n + TB - 1) / TB;
  std::vector<int4> all;
  std::vector<int> off;
  schedule_tasks(MT, NTt, g, all, off);
  if (offsets)
    for (size_t k = 0; k < off.size(); ++k) offsets[k] = off[k];
  if (tasks) {
    const int64_t nwrite = std::min<int64_t>(cap, (int64_t)all.size());
    for (int64_t i = 0; i < nwrite; ++i) {
      tasks[4 * i + 0] = all[i].x;
      tasks[4 * i + 1] = all[i].y;
      tasks[4 * i + 2] = all[i].z;
      tasks[4 * i + 3] = all[i].w;
    }
  }
  return (int64_t)all.size();
}

int64_t gptq2d_schedule_sweeps(int m, int n, int32_t* rows, int64_t cap) {
  if (m < 1 || n < 1 || m > 65536 || n > 65536 || cap < 0) {
    set_error("bad shape or capacity");
    return -1;
  }
  const int MT = (m + TB - 1) / TB, NTt = (n + TB - 1) / TB, S = MT + NTt - 1;
  if (rows)
    for (int k = 0; k < S && k < cap; ++k) stage_rows(MT, NTt, k, rows[2 * k], rows[2 * k + 1]);
  return S;
}

}  // extern "C"
