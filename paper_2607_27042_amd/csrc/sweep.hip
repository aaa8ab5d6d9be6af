// The GPTQ-2D rounding sweep on 64 x 64 tiles (Sec. 4.2-4.3).
//
// Tile (I, J) holds rows 64I.. and columns 64J.. of X. An error at (i, j)
// reaches only rows >= i and columns >= j (Eq. rank-one-update), so tiles on
// one tile anti-diagonal I + J = s are independent and are swept together in
// launch s (s = 0 .. MT + NT - 2). Inside a tile the workgroup runs
// Algorithm 3 restricted to the tile; everything that crosses a tile edge is
// deferred, as in Algorithm 4's lazy block update, and delivered as dense
// products on MFMA:
//   down : P[I'][J] += L[I'][I]  E[I][J]      (completes C = L E below, and Y)
//   right: R[I][J'] += C[I][J]  U[J][J']      (right pushes of C = L E)
// With P the accumulated down feedback and R the accumulated right feedback,
// the corrected value of entry (i, j) when it is rounded is
//   y = X + R + (P + in-tile pushes down) + in-tile pushes right,
// which equals X + (L E U)_ij over earlier entries (proof of Theorem 2).
//
// Delivery: the sweeping workgroup of tile (I, J) itself pulls the
// contributions of its two immediate predecessors (I-1, J) and (I, J-1)
// (rank-64 products); everything older is delivered by GEMM tasks that run in
// the same launches as the sweeps, batched over g consecutive tile
// anti-diagonals (rank up to 64 g), never later than the launch before the
// target is swept. Each (target, direction) gets at most one task per launch,
// so accumulation needs no atomics and the result is deterministic.
#include <math.h>

#include <algorithm>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace g2d {

struct StageArgs {
  int m, n, mp, np, MT, NT;
  const double* L;
  const double* U;
  const double* dL;
  const double* dU;
  const void* X;
  int64_t ldx;
  int32_t* Z;
  int64_t ldz;
  void* Y;
  int64_t ldy;
  double* P;
  double* R;
  double* E;
  double* C;
  double* objp;
  int* flags;
  const int4* tasks;
  int stage, ilo, nsweep;
};

struct SweepSmem {
  double LsT[TB + 1][TB];     // LsT[x][r] = L_II[r][x]; row 64 is zero
  double Us[TB + 1][TB + 2];  // Us[y][k] = U_JJ[y][k]; row 64 is zero
  double ev[2][TB];           // error of the active entry of column k
  double cv[2][TB];           // C value of the active entry of row r
  union {
    double T[TB][TB + 1];
    GemmSmem g;
  } x;
  double red[NT];
};

union StageSmem {
  SweepSmem s;
  GemmSmem g;
};

template <typename T>
__device__ __forceinline__ double load_x(const T* X, int64_t ldx, int gi, int gj, int m, int n) {
  return (gi < m && gj < n) ? (double)X[(int64_t)gi * ldx + gj] : 0.0;
}

// One deferred-feedback delivery (a GEMM task).
__device__ void run_task(const StageArgs& a, int4 tk, GemmSmem& sm) {
  const int dir = tk.x & 1, ow = (tk.x >> 1) & 1;
  const int ti = tk.y, tj = tk.z, s0 = tk.w & 0xffff, s1 = tk.w >> 16;
  const int K = (s1 - s0) * TB;
  Acc acc;
  acc.zero();
  double* out;
  if (dir == 0) {
    gemm_acc(acc, OpRK{a.L + (int64_t)ti * TB * a.mp + (int64_t)s0 * TB, a.mp},
             OpKR{a.E + (int64_t)s0 * TB * a.np + (int64_t)tj * TB, a.np}, K, sm);
    out = a.P + (int64_t)ti * TB * a.np + (int64_t)tj * TB;
  } else {
    gemm_acc(acc, OpRK{a.C + (int64_t)ti * TB * a.np + (int64_t)s0 * TB, a.np},
             OpKR{a.U + (int64_t)s0 * TB * a.np + (int64_t)tj * TB, a.np}, K, sm);
    out = a.R + (int64_t)ti * TB * a.np + (int64_t)tj * TB;
  }
  if (!ow) acc_add_from(acc, out, a.np);
  acc_store(acc, out, a.np, 1.0);
}

// Sweep of one tile. Thread layout: wave w, lane l; q = 4w + (l >> 4) picks
// columns 4q .. 4q+3 and p = l & 15 rows 4p .. 4p+3; each thread keeps its
// 4 x 4 block of the tile in registers.
template <typename T>
__device__ void run_sweep(const StageArgs& a, int I, int J, SweepSmem& sm) {
  const int t = threadIdx.x;
  const int q = 4 * (t >> 6) + ((t & 63) >> 4);
  const int p = t & 15;
  const int r0 = 4 * p, k0 = 4 * q;
  const int gi0 = I * TB, gj0 = J * TB;

  // diagonal factor blocks into LDS; zero rows for out-of-tile indices
  for (int e = t; e < TB * TB; e += NT) {
    const int r = e >> 6, x = e & 63;
    sm.LsT[x][r] = a.L[(int64_t)(gi0 + r) * a.mp + gi0 + x];
    sm.Us[r][x] = a.U[(int64_t)(gj0 + r) * a.np + gj0 + x];
  }
  if (t < TB) {
    sm.LsT[TB][t] = 0.0;
    sm.Us[TB][t] = 0.0;
    sm.ev[0][t] = sm.ev[1][t] = 0.0;
    sm.cv[0][t] = sm.cv[1][t] = 0.0;
  }

  double Dn[4][4], Rt[4][4];
  // down feedback: P (older tiles above) + L[I][I-1] E[I-1][J]
  {
    Acc acc;
    acc.zero();
    if (I >= 1)
      gemm_acc(acc, OpRK{a.L + (int64_t)gi0 * a.mp + (int64_t)(gi0 - TB), a.mp},
               OpKR{a.E + (int64_t)(gi0 - TB) * a.np + gj0, a.np}, TB, sm.x.g);
    if (I >= 2) acc_add_from(acc, a.P + (int64_t)gi0 * a.np + gj0, a.np);
    acc_to_lds<TB + 1>(acc, sm.x.T);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Dn[i][j] = sm.x.T[r0 + i][k0 + j];
    __syncthreads();
  }
  // right feedback: R (older tiles to the left) + C[I][J-1] U[J-1][J], plus X
  {
    Acc acc;
    acc.zero();
    if (J >= 1)
      gemm_acc(acc, OpRK{a.C + (int64_t)gi0 * a.np + (int64_t)(gj0 - TB), a.np},
               OpKR{a.U + (int64_t)(gj0 - TB) * a.np + gj0, a.np}, TB, sm.x.g);
    if (J >= 2) acc_add_from(acc, a.R + (int64_t)gi0 * a.np + gj0, a.np);
    acc_to_lds<TB + 1>(acc, sm.x.T);
    __syncthreads();
    const T* X = (const T*)a.X;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        Rt[i][j] = sm.x.T[r0 + i][k0 + j] + load_x<T>(X, a.ldx, gi0 + r0 + i, gj0 + k0 + j, a.m, a.n);
    __syncthreads();
  }

  // In-tile Algorithm 3. Stage d handles the entries with r + k == d. The
  // window Lw[x & 3][i] holds L[r0+i][x] for x = d-k0-3 .. d-k0 and
  // Uw[y & 3][j] holds U[y][k0+j] for y = d-r0-3 .. d-r0.
  double yf[4][4], cf[4][4], Lw[4][4], Uw[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      Lw[i][j] = 0.0;
      Uw[i][j] = 0.0;
      yf[i][j] = 0.0;
      cf[i][j] = 0.0;
    }
  const int pq = p + q;
  for (int D = 0; D < TB / 2; ++D) {
#pragma unroll
    for (int dl = 0; dl < 4; ++dl) {
      const int d = 4 * D + dl;
      if (d <= 2 * TB - 2) {
        int x = d - k0;
        x = (x < 0 || x >= TB) ? TB : x;
        int y = d - r0;
        y = (y < 0 || y >= TB) ? TB : y;
#pragma unroll
        for (int i = 0; i < 4; ++i) Lw[dl][i] = sm.LsT[x][r0 + i];
#pragma unroll
        for (int j = 0; j < 4; ++j) Uw[dl][j] = sm.Us[y][k0 + j];
        const int buf = dl & 1;
        // round the entries of this thread's block that lie on anti-diagonal d
#pragma unroll
        for (int grp = 0; grp < 2; ++grp) {
          if (D == pq + grp) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int j = dl + 4 * grp - i;
              if (j >= 0 && j < 4) {
                const double yv = Rt[i][j] + Dn[i][j];
                const double z = rint(yv);
                const double e = z - yv;
                const double c = Dn[i][j] + e;
                yf[i][j] = yv;
                cf[i][j] = c;
                sm.ev[buf][k0 + j] = e;
                sm.cv[buf][r0 + i] = c;
              }
            }
          }
        }
        __syncthreads();
        double e4[4], c4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) e4[j] = sm.ev[buf][k0 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i) c4[i] = sm.cv[buf][r0 + i];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            Dn[i][j] += Lw[(dl - j) & 3][i] * e4[j];  // push down
            Rt[i][j] += c4[i] * Uw[(dl - i) & 3][j];  // push right
          }
      }
    }
  }

  // outputs
  double part = 0.0;
  int bad = 0;
  T* Y = (T*)a.Y;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int gi = gi0 + r0 + i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gj = gj0 + k0 + j;
      const double yv = yf[i][j];
      const double z = rint(yv);
      const double e = z - yv;
      a.E[(int64_t)gi * a.np + gj] = e;
      a.C[(int64_t)gi * a.np + gj] = cf[i][j];
      if (gi < a.m && gj < a.n) {
        if (!isfinite(yv)) bad |= FLAG_NONFINITE;
        else if (fabs(z) > 2147483647.0) bad |= FLAG_OVERFLOW;
        const double zc = fmin(fmax(z, -2147483648.0), 2147483647.0);
        a.Z[(int64_t)gi * a.ldz + gj] = isfinite(zc) ? (int32_t)zc : 0;
        if (Y) Y[(int64_t)gi * a.ldy + gj] = (T)yv;
        part += e * e * a.dL[gi] * a.dU[gj];
      }
    }
  }
  if (bad) raise_flag(a.flags, bad);
  sm.red[t] = part;
  __syncthreads();
  if (t == 0) {
    double s = 0.0;
    for (int i = 0; i < NT; ++i) s += sm.red[i];
    a.objp[I * a.NT + J] = s;
  }
}

template <typename T>
__global__ __launch_bounds__(NT) void k_stage(StageArgs a) {
  __shared__ StageSmem sm;
  const int b = blockIdx.x;
  if (b < a.nsweep) {
    const int I = a.ilo + b;
    run_sweep<T>(a, I, a.stage - I, sm.s);
  } else {
    run_task(a, a.tasks[b - a.nsweep], sm.g);
  }
}

__global__ __launch_bounds__(NT) void k_obj_reduce(const double* part, int count, double* out) {
  __shared__ double red[NT];
  double s = 0.0;
  for (int i = threadIdx.x; i < count; i += NT) s += part[i];
  red[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int i = 0; i < NT; ++i) tot += red[i];
    out[0] = tot;
  }
}

__global__ void k_zero_flags(int* p) {
  if (threadIdx.x == 0) p[0] = 0;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

size_t workspace_bytes(const Factors& f) {
  const size_t tile = (size_t)f.mp * f.np * sizeof(double);
  size_t objp = ((size_t)f.MT * f.NT * sizeof(double) + 255) / 256 * 256;
  return 256 + objp + 4 * tile;
}

Workspace workspace_carve(const Factors& f, void* base) {
  char* p = (char*)base;
  Workspace w;
  w.flags = (int*)p;
  p += 256;
  w.objp = (double*)p;
  p += ((size_t)f.MT * f.NT * sizeof(double) + 255) / 256 * 256;
  const size_t tile = (size_t)f.mp * f.np * sizeof(double);
  w.P = (double*)p;
  w.R = (double*)(p + tile);
  w.E = (double*)(p + 2 * tile);
  w.C = (double*)(p + 3 * tile);
  return w;
}

void schedule_tasks(int MT, int NTt, int g, std::vector<int4>& all, std::vector<int>& off) {
  const int S = MT + NTt - 1;
  if (g < 1) g = 1;
  std::vector<std::vector<int4>> per(S);
  for (int ti = 0; ti < MT; ++ti) {
    for (int tj = 0; tj < NTt; ++tj) {
      const int sig = ti + tj;
      if (sig < 2) continue;
      for (int dir = 0; dir < 2; ++dir) {
        const int fixed = dir == 0 ? tj : ti;  // source stage = source index + fixed
        const int lim = dir == 0 ? ti - 2 : tj - 2;
        if (lim < 0) continue;
        bool first = true;
        auto add = [&](int launch, int lo, int hi) {
          const int s0 = std::max(lo - fixed, 0), s1 = std::min(hi - fixed, lim) + 1;
          if (s1 <= s0) return;
          const int ow = first ? 1 : 0;
          first = false;
          per[launch].push_back(make_int4(dir | (ow << 1), ti, tj, s0 | (s1 << 16)));
        };
        // whole batches of g source anti-diagonals, spread over the g launches
        // after the batch completes, each at least one launch before the target
        for (int beta = 0; (beta + 1) * g <= sig - 2; ++beta) {
          const int launch = (beta + 1) * g + ((sig - (beta + 1) * g - 2) % g);
          add(launch, beta * g, beta * g + g - 1);
        }
        // the rest, in the launch just before the target is swept
        add(sig - 1, g * ((sig - 2) / g), sig - 2);
      }
    }
  }
  all.clear();
  off.assign(S + 1, 0);
  for (int k = 0; k < S; ++k) {
    std::stable_sort(per[k].begin(), per[k].end(), [](const int4& x, const int4& y) {
      return ((x.w >> 16) - (x.w & 0xffff)) > ((y.w >> 16) - (y.w & 0xffff));
    });
    off[k] = (int)all.size();
    all.insert(all.end(), per[k].begin(), per[k].end());
  }
  off[S] = (int)all.size();
}

gptq2d_status build_schedule(Factors& f, int g) {
  std::vector<int4> all;
  std::vector<int> off;
  if (g < 1) g = 1;
  schedule_tasks(f.MT, f.NT, g, all, off);
  if (f.sched.d_tasks) {
    (void)hipFree(f.sched.d_tasks);
    f.sched.d_tasks = nullptr;
  }
  if (!all.empty()) {
    hipError_t e = hipMalloc(&f.sched.d_tasks, all.size() * sizeof(int4));
    if (e != hipSuccess) return hip_fail(e, "schedule allocation");
    e = hipMemcpy(f.sched.d_tasks, all.data(), all.size() * sizeof(int4), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "schedule upload");
  }
  f.sched.g = g;
  f.sched.stages = f.MT + f.NT - 1;
  f.sched.offset = off;
  f.sched.ntasks = all.size();
  return GPTQ2D_OK;
}

template <typename T>
static gptq2d_status round_typed(const Factors& f, const void* X, int64_t ldx, int32_t* Z,
                                 int64_t ldz, void* Y, int64_t ldy, double* objective,
                                 const Workspace& ws, hipStream_t s) {
  StageArgs a;
  a.m = f.m;
  a.n = f.n;
  a.mp = f.mp;
  a.np = f.np;
  a.MT = f.MT;
  a.NT = f.NT;
  a.L = f.L;
  a.U = f.U;
  a.dL = f.dL;
  a.dU = f.dU;
  a.X = X;
  a.ldx = ldx;
  a.Z = Z;
  a.ldz = ldz;
  a.Y = Y;
  a.ldy = ldy;
  a.P = ws.P;
  a.R = ws.R;
  a.E = ws.E;
  a.C = ws.C;
  a.objp = ws.objp;
  a.flags = ws.flags;
  hipLaunchKernelGGL(k_zero_flags, dim3(1), dim3(64), 0, s, ws.flags);
  const Schedule& S = f.sched;
  for (int k = 0; k < S.stages; ++k) {
    const int ilo = std::max(0, k - (f.NT - 1)), ihi = std::min(k, f.MT - 1);
    a.stage = k;
    a.ilo = ilo;
    a.nsweep = ihi - ilo + 1;
    const int ntasks = S.offset[k + 1] - S.offset[k];
    a.tasks = S.d_tasks ? S.d_tasks + S.offset[k] : nullptr;
    hipLaunchKernelGGL(k_stage<T>, dim3(a.nsweep + ntasks), dim3(NT), 0, s, a);
  }
  if (objective)
    hipLaunchKernelGGL(k_obj_reduce, dim3(1), dim3(NT), 0, s, ws.objp, f.MT * f.NT, objective);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "sweep launch");
  return GPTQ2D_OK;
}

gptq2d_status launch_round(const Factors& f, gptq2d_dtype dt, const void* X, int64_t ldx,
                           int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                           const Workspace& ws, hipStream_t s) {
  if (dt == GPTQ2D_F32) return round_typed<float>(f, X, ldx, Z, ldz, Y, ldy, objective, ws, s);
  return round_typed<double>(f, X, ldx, Z, ldz, Y, ldy, objective, ws, s);
}

}  // namespace g2d
