// Internal declarations of the GPTQ-2D library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "gptq2d.h"

namespace g2d {

// Deferred-feedback delivery of the blocked sweep: one GEMM task that adds the
// contribution of a contiguous run of finished source tiles to a block of up
// to 2 x 2 target tiles. x = dir | overwrite << 1 | (rows - 1) << 2 |
// (cols - 1) << 3, y = first target tile row, z = first target tile column,
// w = first source | (one past last source) << 16.
struct Schedule {
  int g = 0;                     // batch width in tile anti-diagonals
  int stages = 0;                // tile anti-diagonals: MT + NT - 1
  std::vector<int> offset;       // per stage: first task (size stages + 1)
  std::vector<int> bin_offset;   // per stage: first bin (size stages + 1)
  int4* d_tasks = nullptr;       // all tasks, grouped by stage, then by bin
  int4* d_bins = nullptr;        // {first task in the stage, counts by shape}, grouped by stage
  int4* d_stage = nullptr;       // per stage: {offset, bin_offset, bins, 0} (batched rounding)
  void* d_base = nullptr;        // the handle's fixed stage arguments on the device (batched rounding)
  size_t ntasks = 0;
};

struct Factors {
  int m = 0, n = 0;     // problem shape
  int mp = 0, np = 0;   // padded to multiples of 64
  int MT = 0, NT = 0;   // tile counts
  int device = 0;
  // rounding order: 0 from the first row and column on, 1 from the last (the
  // factors are then those of the index-reversed problem)
  int rev = 0;
  // outputs of the factorisation (fp64, padded with an identity block)
  double* L = nullptr;   // mp x mp, tile by tile in S order; unit lower; upper tiles not kept
  double* U = nullptr;   // np x np, tile by tile in R order; unit upper; lower tiles not kept
  double* dL = nullptr;  // mp: 1 / lamL
  double* dU = nullptr;  // np: 1 / lamU
  // factorisation scratch, one set per side
  double* gram[2] = {nullptr, nullptr};  // reversed Gram, then its Cholesky factor
  double* inv[2] = {nullptr, nullptr};   // inverse of that Cholesky factor
  double* dinv[2] = {nullptr, nullptr};  // inverses of its 64 x 64 diagonal blocks
  int* flags = nullptr;                  // device error bits of the factorisation
  double* gpart = nullptr;               // partial Gram tiles split between work groups
  int* genv = nullptr;                   // Gram envelopes and the Gram work plan built from them
  int cus = 256;                         // compute units of the device
  // second stream of the factorisation: the far part of each group's
  // trailing update runs there, next to the following group's panels
  hipStream_t aux = nullptr;
  hipEvent_t ev_near = nullptr, ev_far = nullptr, ev_far1 = nullptr;
  // stream of this handle's factorisation inside a batched call (created on
  // first use) and the event that marks its end
  hipStream_t own = nullptr;
  hipEvent_t ev_own = nullptr;
  Schedule sched;
  // launch timing of the sweep's stage kernel (diagnostics): while enabled,
  // every stage launch records its start and end time stamps into a pair of
  // events; the pairs accumulate until they are read
  bool stage_timing = false;
  mutable std::vector<hipEvent_t> stage_ev;  // event pool, grows on demand
  mutable size_t stage_ev_used = 0;          // events recorded since the last read
  // the handle's fixed factorisation arguments on the device (batched
  // factorisation), fac_static_bytes() bytes
  void* d_fac = nullptr;
  std::vector<void*> allocations;
};

// workspace layout of gptq2d_round
struct Workspace {
  int* flags;
  double* objp;  // per-tile objective partials, MT x NT
  double* P;     // deferred down feedback (rows below), mp x np
  double* R;     // deferred right feedback (columns to the left), mp x np
  double* E;     // rounding errors, mp x np
  double* C;     // the buffer C = L E, mp x np
};
// the layout itself, on the host and on the device (a batched sweep finds
// each problem's buffers in its workspace region)
__host__ __device__ inline Workspace carve_workspace(void* base, int mp, int np, int MT, int NT) {
  char* p = (char*)base;
  Workspace w;
  w.flags = (int*)p;
  p += 256;
  w.objp = (double*)p;
  p += ((size_t)MT * NT * sizeof(double) + 255) / 256 * 256;
  const size_t tile = (size_t)mp * np * sizeof(double);
  w.P = (double*)p;
  w.R = (double*)(p + tile);
  w.E = (double*)(p + 2 * tile);
  w.C = (double*)(p + 3 * tile);
  return w;
}
size_t workspace_bytes(const Factors& f);

// The tiles swept by launch k of the sweep (Fig. 1 at tile level: the tile
// anti-diagonal I + J = k): tile rows ilo .. ihi, tile (I, k - I) each.
__host__ __device__ inline void stage_rows(int MT, int NT, int k, int& ilo, int& ihi) {
  ilo = k - (NT - 1) > 0 ? k - (NT - 1) : 0;
  ihi = k < MT - 1 ? k : MT - 1;
}
Workspace workspace_carve(const Factors& f, void* base);

// status plumbing
void set_error(const std::string& msg);
gptq2d_status hip_fail(hipError_t e, const char* what);
// the handle's device is the current one
gptq2d_status check_device(const Factors* f);
// the arguments gptq2d_round checks before its workspace
gptq2d_status check_round_args(const Factors* f, gptq2d_dtype dt, const void* X, int64_t ldx,
                               const int32_t* Z, int64_t ldz, const void* Y, int64_t ldy);

// factorisation launches (enqueued on stream, no synchronisation)
// doubles of scratch for the Gram tiles split between work groups
size_t gram_part_doubles(int m, int n, int cus);
size_t gram_env_ints(int m, int n);
// stream-ordered upload of host words into device memory (bytes and dst
// multiples of 8; the host buffer may be reused on return)
gptq2d_status enqueue_upload(void* dst, const void* src, size_t bytes, hipStream_t s);
// batched factorisation of problems of one shape (fs[0]'s second stream and
// events order it); `table` holds factor_batch_table_bytes(count) bytes of
// device memory
size_t factor_batch_table_bytes(int count);
// the handle's fixed factorisation arguments, copied to f.d_fac (synchronous)
size_t fac_static_bytes();
gptq2d_status upload_fac_static(Factors& f);
gptq2d_status launch_factor_batched(int count, Factors* const* fs, gptq2d_dtype dt,
                                    const void* const* A, const int64_t* lda, const void* const* B,
                                    const int64_t* ldb, void* table, hipStream_t s);
gptq2d_status launch_factor(Factors& f, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, hipStream_t s);
gptq2d_status launch_export(const Factors& f, double* L, int64_t ldl, double* U, int64_t ldu,
                            double* lamL, double* lamU, hipStream_t s);
gptq2d_status launch_import(Factors& f, const double* L, int64_t ldl, const double* U,
                            int64_t ldu, const double* lamL, const double* lamU, hipStream_t s);

// sweep
void schedule_tasks(int MT, int NT, int g, std::vector<int4>& all, std::vector<int>& offset);
// Packs each stage's tasks into bins (one work group each) for `units`
// compute units; reorders `all` within every stage.
gptq2d_status pack_bins(int MT, int NT, int units, std::vector<int4>& all,
                        const std::vector<int>& offset, std::vector<int4>& bins,
                        std::vector<int>& bin_offset);
gptq2d_status build_schedule(Factors& f, int g);
void free_schedule(Schedule& s);
// allow_timing = false: no stage-launch timing even if the handle asks for it
// (timing creates HIP events on first use)
gptq2d_status launch_round(const Factors& f, gptq2d_dtype dt, const void* X, int64_t ldx,
                           int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                           const Workspace& ws, hipStream_t s, bool allow_timing = true);

// batched rounding: `count` problems, one workspace region each, in common
// stage launches (workspace layout in sweep.hip)
size_t batched_workspace_bytes(int count, const Factors* const* f);
gptq2d_status launch_round_batched(int count, const Factors* const* f, gptq2d_dtype dt,
                                   const void* const* X, const int64_t* ldx, int32_t* const* Z,
                                   const int64_t* ldz, void* const* Y, const int64_t* ldy,
                                   double* objective, void* workspace, hipStream_t s);

}  // namespace g2d

// the opaque handle of the C ABI is the factor record itself
struct gptq2d_factors_s : g2d::Factors {};
