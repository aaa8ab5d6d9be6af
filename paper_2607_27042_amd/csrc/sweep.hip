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
#include <hip/hip_ext.h>
#include <math.h>

#include <algorithm>
#include <cstring>
#include <functional>
#include <queue>
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
  // X, Z, Y at element (i, j) of the problem the sweep runs on: base + i ld +
  // j cstep. In the forward order cstep = 1 and the bases are the matrices';
  // in reverse order the problem is the index-reversed one, so each base is
  // the matrix's last element, ld its negated row stride and cstep = -1.
  const void* X;
  int64_t ldx;
  int32_t* Z;
  int64_t ldz;
  void* Y;
  int64_t ldy;
  int cstep;
  double* P;
  double* R;
  double* E;
  double* C;
  double* objp;
  int* flags;
  const int4* tasks;  // this launch's deliveries, grouped by bin
  const int4* bins;   // this launch's bins (one work group each)
  int stage, ilo, nsweep;
  // batched rounding: the problem's per-stage table {first task, first bin,
  // bins, 0}; tasks and bins then point at the problem's whole plan
  const int4* stab;
};

constexpr int SS = 16;       // sub-tile edge of the in-tile sweep
constexpr int TP = TB + 2;   // LDS row stride of the tile arrays (doubles)

// LDS of a sweeping workgroup. Ls, Us: the diagonal factor blocks L_II and
// U_JJ with zero columns 64, 65 (Ls) and zero rows 64, 65 (Us) for source
// blocks that do not exist. Et, Ct: the tile's E and C as its sub-tiles finish (the
// operands of the in-tile feedback products); before the sweep the same bytes
// stage the two neighbour products.
struct SweepSmem {
  double Ls[TB][TP];
  double Us[TB + 2][TP];
  union {
    struct {
      double Et[TB][TP];
      double Ct[TB][TP];
    } t;
    Stage64 g;
    double T[TB][TB + 1];
  } x;
  double scr[4][SS][SS + 1]; // per wave: MFMA-layout to block-layout transfer
  double red[NT / 64];
  int done[4];               // per wave: sub-tiles finished (release/acquire, workgroup scope)
};

// Staging of one 32-deep chunk of a delivery product, filled by direct
// global -> LDS loads (each wave instruction moves 64 lanes x 16 bytes to 1 KB
// of consecutive LDS): the left operand in blocks of four rows, each row's
// 16-byte pieces permuted by an XOR with the row's position in the block and
// every block padded by 64 bytes (an MFMA operand read of 16 rows then hits 16
// distinct bank groups), the right operand as rows b[k][col] padded to 130
// doubles. With the tile-contiguous storage a left-operand load reads 1 KB of
// contiguous memory and a right-operand load two 512-byte runs.
constexpr int KQ = 32;
constexpr int AQ = 4 * KQ + 8;  // doubles per 4-row block of the left operand (64 B pad)
struct TaskChunk {
  double a[2 * TB / 4][AQ];
  double b[KQ][2 * TB + 2];
};
struct TaskSmem {
  TaskChunk buf[2];
};

union StageSmem {
  SweepSmem s;
  TaskSmem t;
};

// X[gi][gj] widened, 0 outside the matrix; the load is unconditional (from a
// clamped address) so that it does not serialise behind a branch.
template <typename T>
__device__ __forceinline__ double load_x(const T* X, int64_t ldx, int cstep, int gi, int gj, int m,
                                         int n) {
  const bool ok = gi < m && gj < n;
  const T v = X[ok ? (int64_t)gi * ldx + gj * cstep : 0];
  return ok ? (double)v : 0.0;
}

// Operands of one delivery (uniform over the work group): out (+)= A B with
// A the (64 nr) x (64 K) source panel and B the (64 K) x (64 nc) panel, all
// tile-contiguous: A points at its first tile (S order), the next tile row
// ars doubles on and the next source tile 4096 on; B at its first tile (R
// order), the next source tile row bks on and the next tile column 4096 on;
// out at the first target tile (R order), the next tile row ors on.
struct TaskOp {
  const double* A;
  const double* B;
  double* out;
  int64_t ars, bks, ors;
  int nch, ow, nr, nc;
};

__device__ __forceinline__ TaskOp task_op(const StageArgs& a, int4 tk) {
  const int dir = tk.x & 1;
  const int ti = tk.y, tj = tk.z, s0 = tk.w & 0xffff, s1 = tk.w >> 16;
  TaskOp T;
  T.ow = (tk.x >> 1) & 1;
  T.nr = ((tk.x >> 2) & 1) + 1;
  T.nc = ((tk.x >> 3) & 1) + 1;
  T.nch = (s1 - s0) * (TB / KQ);
  T.bks = tile_off(1, 0, a.NT);
  T.ors = tile_off(1, 0, a.NT);
  if (dir == 0) {
    T.A = a.L + tile_off(ti, s0, a.MT);
    T.ars = tile_off(1, 0, a.MT);
    T.B = a.E + tile_off(s0, tj, a.NT);
    T.out = a.P + tile_off(ti, tj, a.NT);
  } else {
    T.A = a.C + tile_off(ti, s0, a.NT);
    T.ars = tile_off(1, 0, a.NT);
    T.B = a.U + tile_off(s0, tj, a.NT);
    T.out = a.R + tile_off(ti, tj, a.NT);
  }
  return T;
}

typedef __attribute__((address_space(3))) void lds_void;

// Chunk c of task T into d (source tile c / 2, its columns (rows of B)
// 32 (c % 2) ..): wave w moves the left-operand row blocks j = w + 4i (rows
// 4j .. 4j+3, i < 4 nr: 1 KB of contiguous memory in S order) and the
// right-operand rows k = w + 4i (i < 8), each a 1 KB direct global -> LDS
// load. Lane l of a left-operand load takes the 16-byte piece
// (l & 15) ^ (l >> 4) of row 4j + (l >> 4); of a right-operand load the
// columns 2l, 2l+1 (clamped to the target: never used past it).
// (i0, i1 select the part i0 <= i < i1 of the loads)
__device__ __forceinline__ void task_issue(const TaskOp& T, int c, TaskChunk& d, int w, int l, int i0 = 0,
                                           int i1 = 8) {
  const int ar = l >> 4, ap = (l & 15) ^ ar;
  const double* ac = T.A + (int64_t)(c >> 1) * 4096 + (c & 1) * 2048;
  const int col = min(2 * l, TB * T.nc - 2);
  const double* pb = T.B + (int64_t)(c >> 1) * T.bks + (c & 1) * 32 * TB + (col >> 6) * 4096 + (col & 63);
#pragma unroll
  for (int i = i0; i < i1; ++i) {
    const int j = w + 4 * i;
    if (i < 4 * T.nr) {
      const double* pa = ac + (j >> 4) * T.ars + (4 * (j & 15) + ar) * 32 + 2 * ap;
      __builtin_amdgcn_global_load_lds((const void*)pa, (lds_void*)&d.a[j][0], 16, 0, 0);
    }
    __builtin_amdgcn_global_load_lds((const void*)(pb + j * TB), (lds_void*)&d.b[j][0], 16, 0, 0);
  }
}

// The part of a (64 nr) x (64 nc) target that wave w computes, as NI x NJ
// MFMA blocks of 16 x 16 from row rb and column cb:
//   2 x 2 tiles: 64 x 64 quadrant (w >> 1, w & 1)      NI = NJ = 4
//   2 x 1 tiles: rows 32 w .. 32 w + 31, all 64 columns NI = 2, NJ = 4
//   1 x 2 tiles: all 64 rows, columns 32 w .. 32 w + 31 NI = 4, NJ = 2
//   1 x 1 tile : 32 x 32 quadrant (w >> 1, w & 1)      NI = NJ = 2
__device__ __forceinline__ void task_part(const TaskOp& T, int w, int& rb, int& cb) {
  if (T.nr == 2 && T.nc == 2) { rb = 64 * (w >> 1); cb = 64 * (w & 1); }
  else if (T.nr == 2) { rb = 32 * w; cb = 0; }
  else if (T.nc == 2) { rb = 0; cb = 32 * w; }
  else { rb = 32 * (w >> 1); cb = 32 * (w & 1); }
}

// Accumulators of the wave's part: the old target values (a delivery that
// adds) or zero (one that overwrites).
// Entry (row, col) of a target (rows and columns counted from its first
// tile) relative to T.out.
__device__ __forceinline__ int64_t task_at(const TaskOp& T, int row, int col) {
  return (row >> 6) * T.ors + (col >> 6) * 4096 + r_idx(row & 63, col & 63);
}

template <int NI, int NJ>
__device__ __forceinline__ void task_init(d4 (&acc)[4][4], const TaskOp& T, int rb, int cb, int l) {
  if (!T.ow) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[i][j][r] = T.out[task_at(T, rb + 16 * i + 4 * r + (l >> 4), cb + 16 * j + (l & 15))];
    // the accumulators are complete before the chunk loop (so that no wait
    // for them lands inside it, where it would also wait for the next chunk)
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  } else {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};
  }
}

template <int NI, int NJ>
__device__ __forceinline__ void task_store(const d4 (&acc)[4][4], const TaskOp& T, int rb, int cb,
                                           int l) {
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        T.out[task_at(T, rb + 16 * i + 4 * r + (l >> 4), cb + 16 * j + (l & 15))] = acc[i][j][r];
}

// One staged chunk on MFMA: acc[i][j] += A(rows rb + 16 i ..) B(cols cb + 16 j ..).
// The operands of k-step kk + 1 are read while kk is on MFMA (two register
// sets), the reads spread between the MFMAs; mid() runs half-way (before the
// MFMAs of k-step KQ / 8).
template <int NI, int NJ, typename Mid>
__device__ __forceinline__ void task_mma(d4 (&acc)[4][4], const TaskChunk& st, int rb, int cb, int l,
                                         Mid&& mid) {
  const int r0 = l & 15, rr = r0 & 3;
  double av[2][NI], bv[2][NJ];
#pragma unroll
  for (int kk = -1; kk < KQ / 4; ++kk) {
    const int nx = (kk + 1) & 1;
    if (kk + 1 < KQ / 4) {
      const int k = 4 * (kk + 1) + (l >> 4), kp = 2 * (kk + 1) + (l >> 5), e = (l >> 4) & 1;
      const int ao = KQ * rr + 2 * (kp ^ rr) + e;
#pragma unroll
      for (int i = 0; i < NI; ++i) av[nx][i] = st.a[(rb + 16 * i + r0) >> 2][ao];
#pragma unroll
      for (int j = 0; j < NJ; ++j) bv[nx][j] = st.b[k][cb + 16 * j + r0];
    }
    if (kk == KQ / 8) {
      // half-way: the rest of the next chunk's loads
      __builtin_amdgcn_sched_barrier(0);
      mid();
      __builtin_amdgcn_sched_barrier(0);
    }
    if (kk >= 0) {
      const int cur = kk & 1;
#pragma unroll
      for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[cur][i], bv[cur][j], acc[i][j], 0, 0, 0);
      if (kk + 1 < KQ / 4) {
        constexpr int NM = NI * NJ, NR = NI + NJ;  // MFMAs and reads per k-step
#pragma unroll
        for (int u = 0; u < NR; ++u) {
          __builtin_amdgcn_sched_group_barrier(0x008, NM / NR > 0 ? NM / NR : 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    }
  }
}

// A run of n deliveries of one target shape (NI x NJ blocks per wave),
// streamed through one double-buffered pipeline: the next chunk of a
// delivery is loaded while the current one is on MFMA. At a delivery's end
// its result is stored first, and only then are the next delivery's first
// chunk and old target values loaded: stores queued behind loads wait for
// the memory pipeline, which costs more than the one exposed load latency.
// Every wave has a part of every target (task_part).
template <int NI, int NJ>
__device__ void run_stream(const StageArgs& a, const int4* tk, int n, TaskSmem& sm) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  d4 acc[4][4];
  TaskOp T = task_op(a, tk[0]);
  int rb, cb;
  task_part(T, w, rb, cb);
  task_issue(T, 0, sm.buf[0], w, l);
  task_init<NI, NJ>(acc, T, rb, cb, l);
  int idx = 0, c = 0, p = 0;
  for (;;) {
    const bool last = c + 1 == T.nch;
    // the next chunk's loads go out in two halves, the second one half-way
    // through this chunk's MFMAs (one batch of them stalls this wave's issue
    // until the memory pipeline takes it)
    if (!last) task_issue(T, c + 1, sm.buf[p ^ 1], w, l, 0, 4);
    // chunk c has landed (issued after it: the first half of the next, 8 loads)
    if (!last) __builtin_amdgcn_s_waitcnt(0x0f78);  // vmcnt(8)
    else __builtin_amdgcn_s_waitcnt(0x0f70);        // vmcnt(0)
    // a bare barrier: the wait above already covers this wave's part of
    // chunk c, and a fenced barrier would also wait for the next chunk
    asm volatile("s_barrier" ::: "memory");
    task_mma<NI, NJ>(acc, sm.buf[p], rb, cb, l, [&]() {
      if (!last) task_issue(T, c + 1, sm.buf[p ^ 1], w, l, 4, 8);
    });
    // buffer p is refilled next: every wave's reads of it are complete
    // before the barrier, while the next chunk stays in flight
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    p ^= 1;
    if (last) {
      task_store<NI, NJ>(acc, T, rb, cb, l);
      if (++idx == n) break;
      T = task_op(a, tk[idx]);
      c = 0;
      task_issue(T, 0, sm.buf[p], w, l);
      task_init<NI, NJ>(acc, T, rb, cb, l);
    } else {
      ++c;
    }
  }
}

// One bin of a launch's deliveries, bin = {first task, n22 | n21 << 16,
// n12 | n11 << 16, 0}: the counts of 2 x 2, 2 x 1, 1 x 2 and 1 x 1 targets,
// the tasks grouped in that order; each group is one stream.
__device__ void run_bin(const StageArgs& a, int4 bin, TaskSmem& sm) {
  const int4* tk = a.tasks + bin.x;
  const int n4 = bin.y & 0xffff, n21 = bin.y >> 16, n12 = bin.z & 0xffff, n11 = bin.z >> 16;
  bool busy = false;  // a group before this one used the staging buffers
  if (n4) { run_stream<4, 4>(a, tk, n4, sm); busy = true; }
  tk += n4;
  if (n21) { if (busy) __syncthreads(); run_stream<2, 4>(a, tk, n21, sm); busy = true; }
  tk += n21;
  if (n12) { if (busy) __syncthreads(); run_stream<4, 2>(a, tk, n12, sm); busy = true; }
  tk += n12;
  if (n11) { if (busy) __syncthreads(); run_stream<2, 2>(a, tk, n11, sm); }
}

// acc += A (16 x K) B (K x 16) on MFMA, both operands row-major in LDS with
// row strides lda, ldb; K a compile-time multiple of 4: every operand load is
// issued first.
template <int K>
__device__ __forceinline__ void mma16k(d4& acc, const double* pa, int lda, const double* pb, int ldb) {
  if constexpr (K > 0) {
    const int l = threadIdx.x & 63;
    const double* qa = pa + (l & 15) * lda + (l >> 4);
    const double* qb = pb + (l >> 4) * ldb + (l & 15);
    double av[K / 4], bv[K / 4];
#pragma unroll
    for (int s = 0; s < K / 4; ++s) {
      av[s] = qa[4 * s];
      bv[s] = qb[4 * s * ldb];
    }
#pragma unroll
    for (int s = 0; s < K / 4; ++s) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[s], bv[s], acc, 0, 0, 0);
  }
}

// Per-lane constants of a band sweep.
struct Band {
  int w, l, p, q, br, gi0, gj0;
  double* Et;      // the tile's E (R order) and C (S order)
  double* Ct;
  double l10;      // L[br+1][br]
  double u01[4];   // U[uc+2q][uc+2q+1] of sub-tile c (uc = 16 c)
  double dl[2];    // 1 / lamL of the lane's two rows
  bool interior;   // the whole tile lies inside the matrix
  int32_t* zr[2];  // Z and Y at the lane's two rows, column 2q of the tile
  void* yr[2];
};

// Bounded wait until a band's release counter reaches v (workgroup-scope
// acquire); a wait that runs out raises the time-out flag instead of hanging.
__device__ __forceinline__ void wait_band(const int* done, int v, int& bad) {
  int spins = 0;
  while (__hip_atomic_load(done, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < v) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins > (1 << 22)) {
      bad |= FLAG_TIMEOUT;
      break;
    }
  }
}

// acc += A (16 x K) B (K x 16) on MFMA for a K that is a multiple of 16 known
// only at run time (the wave's band index); operands row-major in LDS.
__device__ __forceinline__ void mma16(d4& acc, const double* pa, int lda, const double* pb, int ldb, int K) {
  const int l = threadIdx.x & 63;
  const double* qa = pa + (l & 15) * lda + (l >> 4);
  const double* qb = pb + (l >> 4) * ldb + (l & 15);
#pragma unroll 1
  for (int k0 = 0; k0 < K; k0 += 16) {
    double av[4], bv[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      av[s] = qa[k0 + 4 * s];
      bv[s] = qb[(k0 + 4 * s) * ldb];
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[s], bv[s], acc, 0, 0, 0);
  }
}

// Sub-tile (w, C) of the band: wait for the band above, add the in-tile
// feedback of the finished sub-tiles above and to the left, run Algorithm 3
// on the 16 x 16 block, publish E and C, write the outputs.
template <typename T, int C>
__device__ __forceinline__ void sub_tile(const StageArgs& a, SweepSmem& sm, const Band& b,
                                         double (&Dc)[2][2], double (&Rc)[2][2], const double (&dc)[2],
                                         double& part, int& bad) {
  const int w = b.w, l = b.l, p = b.p, q = b.q, br = b.br;
  constexpr int uc = SS * C;
  // the band above must have finished sub-tile C
  if (w > 0) wait_band(&sm.done[w - 1], C + 1, bad);
  // feedback from the finished sub-tiles above (same column) and to the left
  // (same band) inside this tile
  {
    d4 aD = {0.0, 0.0, 0.0, 0.0}, aR = {0.0, 0.0, 0.0, 0.0};
    mma16k<SS * C>(aR, &sm.x.t.Ct[SS * w][0], TP, &sm.Us[0][uc], TP);
    mma16(aD, &sm.Ls[SS * w][0], TP, &sm.x.t.Et[0][uc], TP, SS * w);
    double(*sc)[SS + 1] = sm.scr[w];
#pragma unroll
    for (int r = 0; r < 4; ++r) sc[4 * r + (l >> 4)][l & 15] = aD[r];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) Dc[i][j] += sc[2 * p + i][2 * q + j];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int r = 0; r < 4; ++r) sc[4 * r + (l >> 4)][l & 15] = aR[r];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) Rc[i][j] += sc[2 * p + i][2 * q + j];
    __builtin_amdgcn_wave_barrier();
  }

  // Algorithm 3 on the 16 x 16 sub-tile, one 2 x 2 block per lane. The
  // blocks form an 8 x 8 grid swept along its anti-diagonals: block (p, q)
  // is rounded in step p + q (an in-block chain of three entry
  // anti-diagonals). In every step each lane first adds the feedback of the
  // blocks finished in the step before that lie above it in its block column
  // (errors through L, Alg. 3 push down) or left of it in its block row (C
  // through U, push right). Those source blocks are read unconditionally
  // (every LDS word they can reach holds a finite value); a source that does
  // not feed the lane gets a zero weight: the zero column of Ls, the zero rows
  // of Us, or, for the block on the lane's own diagonal, the 2 x 2 diagonal
  // blocks of Ls and Us, which hold zeros during the sweep (their one
  // off-diagonal entry is kept in a register).
  // So a lane's accumulators stop changing after its own step, and every
  // lane runs the rounding chain in every step without a branch: before its
  // step it publishes finite placeholders that nobody reads with a nonzero
  // weight, from its step on the final E and C of its block (read back by
  // the same wave in the next step: LDS is in order within a wave, no
  // barrier). The results of the last step are every lane's final values.
  const double u01 = b.u01[C];
  const double l10 = b.l10;
  const double ul = u01 * l10;
  double* const eown = &sm.x.t.Et[br][uc + 2 * q];
  double* const cown = &sm.x.t.Ct[br][uc + 2 * q];
  // sources at step k: E rows 16 w + 2 (k-1-q) .. +1 at the lane's columns,
  // C columns uc + 2 (k-1-p) .. +1 at the lane's rows (a per-lane base plus
  // a constant offset: no address arithmetic in the steps)
  const double* const pe0 = &sm.x.t.Et[0][0] + (SS * w - 2 - 2 * q) * TP + uc + 2 * q;
  const double* const pc0 = &sm.x.t.Ct[0][0] + br * TP + uc - 2 - 2 * p;
  // weights of step k: L rows br, br+1 at columns SS w - 2 - 2 q + 2 k, and U
  // rows uc - 2 - 2 p + 2 k, +1 at columns uc + 2q, +1; a source that does not
  // feed the lane reads zeros at the same step offset instead: the zero rows
  // 64, 65 of Us for L (the offset runs along columns) and the zero columns
  // 64, 65 of Ls for U (it runs along rows). So a step selects one of two
  // bases per operand and adds a constant.
  const double* const plv = &sm.Ls[br][0] + SS * w - 2 - 2 * q;
  const double* const plz = &sm.Us[TB][0];
  const double* const puv = &sm.Us[0][0] + (uc - 2 - 2 * p) * TP + uc + 2 * q;
  const double* const puz = &sm.Ls[0][TB];
  // the weights of step k do not depend on the sweep: they are read one step
  // ahead, after that step's sources, so that the wait for the sources (the
  // errors and C just written by the step before) covers four reads only
  double2 wl[2][2], wu[2][2];
  auto weights = [&](int k, double2(&l)[2], double2(&u)[2]) {
    const bool vr = (unsigned)(k - 1 - q) < (unsigned)p;  // source block row k-1-q above
    const bool vc = (unsigned)(k - 1 - p) < (unsigned)q;  // source block column k-1-p left
    const double* pl = (vr ? plv : plz) + 2 * k;
    const double* pu = (vc ? puv : puz) + 2 * k * TP;
    l[0] = *reinterpret_cast<const double2*>(pl);
    l[1] = *reinterpret_cast<const double2*>(pl + TP);
    u[0] = *reinterpret_cast<const double2*>(pu);
    u[1] = *reinterpret_cast<const double2*>(pu + TP);
  };
  weights(0, wl[0], wu[0]);
  double yf[2][2], cf[2][2], ef[2][2];
#pragma unroll
  for (int k = 0; k < SS - 1; ++k) {
    const double* pe = pe0 + 2 * k * TP;
    const double* pc = pc0 + 2 * k;
    const double2 e0 = *reinterpret_cast<const double2*>(pe);
    const double2 e1 = *reinterpret_cast<const double2*>(pe + TP);
    const double2 c0 = *reinterpret_cast<const double2*>(pc);
    const double2 c1 = *reinterpret_cast<const double2*>(pc + TP);
    // (LDS serves a wave's requests in order: the weight reads go out right
    // behind the source reads, so that they are done before this step's
    // writes and the next step's source reads)
    __builtin_amdgcn_sched_barrier(0);
    if (k + 1 < SS - 1) weights(k + 1, wl[(k + 1) & 1], wu[(k + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
    const double2 l0 = wl[k & 1][0], l1 = wl[k & 1][1];
    const double2 v0 = wu[k & 1][0], v1 = wu[k & 1][1];
    Dc[0][0] = fma(l0.y, e1.x, fma(l0.x, e0.x, Dc[0][0]));
    Dc[0][1] = fma(l0.y, e1.y, fma(l0.x, e0.y, Dc[0][1]));
    Dc[1][0] = fma(l1.y, e1.x, fma(l1.x, e0.x, Dc[1][0]));
    Dc[1][1] = fma(l1.y, e1.y, fma(l1.x, e0.y, Dc[1][1]));
    Rc[0][0] = fma(c0.y, v1.x, fma(c0.x, v0.x, Rc[0][0]));
    Rc[0][1] = fma(c0.y, v1.y, fma(c0.x, v0.y, Rc[0][1]));
    Rc[1][0] = fma(c1.y, v1.x, fma(c1.x, v0.x, Rc[1][0]));
    Rc[1][1] = fma(c1.y, v1.y, fma(c1.x, v0.y, Rc[1][1]));
    // The in-block chain, with every term that does not wait for this step's
    // errors formed first. With D, R the accumulated feedback and
    // C = D + E (L has a unit diagonal):
    //   y00 = R00 + D00
    //   y01 = R01 + D01 + u01 C00          = k01 + u01 e00
    //   y10 = R10 + D10 + l10 e00          = k10 + l10 e00
    //   y11 = R11 + D11 + l10 e01 + u01 C10
    //       = k11 + u01 l10 e00 + l10 e01 + u01 e10
    const double y00 = Rc[0][0] + Dc[0][0];
    const double k01 = fma(Dc[0][0], u01, Rc[0][1] + Dc[0][1]);
    const double k10 = Rc[1][0] + Dc[1][0];
    const double k11 = fma(Dc[1][0], u01, Rc[1][1] + Dc[1][1]);
    const double e00 = rint(y00) - y00;
    const double y01 = fma(e00, u01, k01);
    const double y10 = fma(e00, l10, k10);
    const double m11 = fma(e00, ul, k11);
    const double e01 = rint(y01) - y01;
    const double e10 = rint(y10) - y10;
    const double y11 = fma(e10, u01, fma(e01, l10, m11));
    const double e11 = rint(y11) - y11;
    const double c00 = Dc[0][0] + e00;
    const double c01 = Dc[0][1] + e01;
    const double c10 = fma(l10, e00, Dc[1][0]) + e10;
    const double c11 = fma(l10, e01, Dc[1][1]) + e11;
    *reinterpret_cast<double2*>(eown) = double2{e00, e01};
    *reinterpret_cast<double2*>(eown + TP) = double2{e10, e11};
    *reinterpret_cast<double2*>(cown) = double2{c00, c01};
    *reinterpret_cast<double2*>(cown + TP) = double2{c10, c11};
    if (k == SS - 2) {
      yf[0][0] = y00; yf[0][1] = y01; yf[1][0] = y10; yf[1][1] = y11;
      cf[0][0] = c00; cf[0][1] = c01; cf[1][0] = c10; cf[1][1] = c11;
      ef[0][0] = e00; ef[0][1] = e01; ef[1][0] = e10; ef[1][1] = e11;
    }
  }

  // hand-off to the band below, then the global outputs
  __hip_atomic_store(&sm.done[w], C + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    *reinterpret_cast<double2*>(b.Et + r_idx(br + i, uc + 2 * q)) = double2{ef[i][0], ef[i][1]};
    *reinterpret_cast<double2*>(b.Ct + s_idx(br + i, uc + 2 * q)) = double2{cf[i][0], cf[i][1]};
  }
  const int64_t cs = a.cstep;
  if (b.interior) {
    // every entry of the tile lies inside the matrix: no bounds checks, and
    // the range check folded into one test per entry (NaN fails it too)
    bool ok = true;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int32_t* zr = b.zr[i] + uc * cs;
      T* yr = b.yr[i] ? (T*)b.yr[i] + uc * cs : nullptr;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const double yv = yf[i][j];
        ok = ok && yv >= -2147483648.5 && yv < 2147483647.5;
        const double zc = fmin(fmax(rint(yv), -2147483648.0), 2147483647.0);
        zr[j * cs] = (int32_t)zc;
        if (yr) yr[j * cs] = (T)yv;
        part = fma(ef[i][j] * ef[i][j], b.dl[i] * dc[j], part);
      }
    }
    if (!ok) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) bad |= isfinite(yf[i][j]) ? 0 : FLAG_NONFINITE;
      if (!(bad & FLAG_NONFINITE)) bad |= FLAG_OVERFLOW;
    }
  } else {
    T* Y = (T*)a.Y;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int gi = b.gi0 + br + i;
      const int gj = b.gj0 + uc + 2 * q;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const double yv = yf[i][j];
        const double z = rint(yv);
        if (gi < a.m && gj + j < a.n) {
          if (!isfinite(yv)) bad |= FLAG_NONFINITE;
          else if (z < -2147483648.0 || z > 2147483647.0) bad |= FLAG_OVERFLOW;
          const double zc = fmin(fmax(z, -2147483648.0), 2147483647.0);
          a.Z[(int64_t)gi * a.ldz + (gj + j) * cs] = isfinite(zc) ? (int32_t)zc : 0;
          if (Y) Y[(int64_t)gi * a.ldy + (gj + j) * cs] = (T)yv;
          part = fma(ef[i][j] * ef[i][j], b.dl[i] * dc[j], part);
        }
      }
    }
  }
}

// Sweep of one tile. Wave w owns the 16-row band 16w .. 16w+15 and sweeps its
// four 16 x 16 sub-tiles left to right, one wave per sub-tile, so that the
// per-anti-diagonal exchange stays inside the wave (LDS, no workgroup
// barrier). Sub-tile (w, c) starts when the band above has finished
// sub-tile c; the feedback from the finished sub-tiles above and to the left
// is added first as two small MFMA products. Lane l owns the 2 x 2 block at
// band rows 2p, 2p+1 (p = l >> 3) and sub-tile columns 2q, 2q+1 (q = l & 7):
// eight consecutive lanes read eight different column pairs of a factor row,
// which keeps the LDS window reads free of bank conflicts.
template <typename T>
__device__ void run_sweep(const StageArgs& a, int I, int J, SweepSmem& sm) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  const int p = l >> 3, q = l & 7;
  const int br = SS * w + 2 * p;  // tile row of the lane's first row
  const int gi0 = I * TB, gj0 = J * TB;
  const T* X = (const T*)a.X;

  // every global load of the prologue is issued before any is used, in the
  // order they are needed: the factor blocks, the operands of the two
  // neighbour products, then X and the accumulated feedback
  double lv[16], uv[16], ga[16], gb[16], gc[16], gd[16];
  load_blk_s(a.L + tile_off(I, I, a.MT), lv);
  load_blk(a.U + tile_off(J, J, a.NT), TB, uv);
  if (I >= 1) {
    load_blk_s(a.L + tile_off(I, I - 1, a.MT), ga);
    load_blk(a.E + tile_off(I - 1, J, a.NT), TB, gb);
  }
  if (J >= 1) {
    load_blk_s(a.C + tile_off(I, J - 1, a.NT), gc);
    load_blk(a.U + tile_off(J - 1, J, a.NT), TB, gd);
  }
  // the off-diagonal entries of the lane's 2 x 2 diagonal factor blocks
  const double l10v = a.L[tile_off(I, I, a.MT) + s_idx(br + 1, br)];
  double u01v[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) u01v[c] = a.U[tile_off(J, J, a.NT) + r_idx(SS * c + 2 * q, SS * c + 2 * q + 1)];
  double Dn[4][2][2], Rt[4][2][2], dl[2], du[4][2];
#pragma unroll
  for (int i = 0; i < 2; ++i) dl[i] = a.dL[gi0 + br + i];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int j = 0; j < 2; ++j) du[c][j] = a.dU[gj0 + SS * c + 2 * q + j];
  // X, then the accumulated right (R, from tile column 2 on) and down (P,
  // from tile row 2 on) feedback; each group is issued as one batch
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        Rt[c][i][j] = load_x<T>(X, a.ldx, a.cstep, gi0 + br + i, gj0 + SS * c + 2 * q + j, a.m, a.n);
  double2 rv[4][2], pv[4][2];
  if (J >= 2) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        rv[c][i] = *reinterpret_cast<const double2*>(a.R + tile_off(I, J, a.NT) + r_idx(br + i, SS * c + 2 * q));
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i) rv[c][i] = double2{0.0, 0.0};
  }
  if (I >= 2) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        pv[c][i] = *reinterpret_cast<const double2*>(a.P + tile_off(I, J, a.NT) + r_idx(br + i, SS * c + 2 * q));
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i) pv[c][i] = double2{0.0, 0.0};
  }
  // the factor blocks go to LDS with their 2 x 2 diagonal blocks zeroed: the
  // block sweep takes the one off-diagonal entry of each (l10, u01) from a
  // register, and the zeros make the lane's own block a zero-weight source
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s, r = e >> 6, x = e & 63;
    const bool dg = (r >> 1) == (x >> 1);
    sm.Ls[r][x] = dg ? 0.0 : lv[s];
    sm.Us[r][x] = dg ? 0.0 : uv[s];
  }
  if (t < TB) {
    *reinterpret_cast<double2*>(&sm.Ls[t][TB]) = double2{0.0, 0.0};
    sm.Us[TB][t] = 0.0;
    sm.Us[TB + 1][t] = 0.0;
  }
  if (t < 4) sm.done[t] = 0;

  // feedback of the neighbouring tiles: L[I][I-1] E[I-1][J] and C[I][J-1]
  // U[J-1][J]; the accumulated feedback (P, R) is added first, as before
  // either product
  Acc acc;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      Dn[c][i][0] = pv[c][i].x;
      Dn[c][i][1] = pv[c][i].y;
    }
  if (I >= 1) {
    acc.zero();
    put_a(sm.x.g, ga);
    put_b(sm.x.g, gb);
    __syncthreads();
    mma_blk(acc, sm.x.g);
    __syncthreads();
    acc_to_lds<TB + 1>(acc, sm.x.T);
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Dn[c][i][j] += sm.x.T[br + i][SS * c + 2 * q + j];
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      Rt[c][i][0] += rv[c][i].x;
      Rt[c][i][1] += rv[c][i].y;
    }
  if (J >= 1) {
    acc.zero();
    __syncthreads();
    put_a(sm.x.g, gc);
    put_b(sm.x.g, gd);
    __syncthreads();
    mma_blk(acc, sm.x.g);
    __syncthreads();
    acc_to_lds<TB + 1>(acc, sm.x.T);
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Rt[c][i][j] += sm.x.T[br + i][SS * c + 2 * q + j];
  }
  __syncthreads();
  // Et / Ct start at zero, their padding columns included: the block sweep
  // reads (zero-weighted) source blocks before they are written, and its
  // C-source reads of the first sub-tile reach back into the padding of the
  // row before; every wave zeroes its band, and the barrier makes the whole
  // arrays zero before any wave sweeps
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int e = l + 64 * s, r = SS * w + (e >> 5), x = 2 * (e & 31);
    *reinterpret_cast<double2*>(&sm.x.t.Et[r][x]) = double2{0.0, 0.0};
    *reinterpret_cast<double2*>(&sm.x.t.Ct[r][x]) = double2{0.0, 0.0};
  }
  if (l < 2 * SS) {
    double(*arr)[TP] = l < SS ? sm.x.t.Et : sm.x.t.Ct;
    *reinterpret_cast<double2*>(&arr[SS * w + (l & (SS - 1))][TB]) = double2{0.0, 0.0};
  }
  Band bd;
  bd.w = w; bd.l = l; bd.p = p; bd.q = q; bd.br = br; bd.gi0 = gi0; bd.gj0 = gj0;
  bd.Et = a.E + tile_off(I, J, a.NT);
  bd.Ct = a.C + tile_off(I, J, a.NT);
  bd.l10 = l10v;
#pragma unroll
  for (int c = 0; c < 4; ++c) bd.u01[c] = u01v[c];
  bd.dl[0] = dl[0];
  bd.dl[1] = dl[1];
  bd.interior = gi0 + TB <= a.m && gj0 + TB <= a.n;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    bd.zr[i] = a.Z + (int64_t)(gi0 + br + i) * a.ldz + (int64_t)(gj0 + 2 * q) * a.cstep;
    bd.yr[i] = a.Y ? (void*)((T*)a.Y + (int64_t)(gi0 + br + i) * a.ldy + (int64_t)(gj0 + 2 * q) * a.cstep)
                   : nullptr;
  }
  __syncthreads();

  double part = 0.0;
  int bad = 0;
  sub_tile<T, 0>(a, sm, bd, Dn[0], Rt[0], du[0], part, bad);
  sub_tile<T, 1>(a, sm, bd, Dn[1], Rt[1], du[1], part, bad);
  sub_tile<T, 2>(a, sm, bd, Dn[2], Rt[2], du[2], part, bad);
  sub_tile<T, 3>(a, sm, bd, Dn[3], Rt[3], du[3], part, bad);

  if (bad) raise_flag(a.flags, bad);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
  if (l == 0) sm.red[w] = part;
  __syncthreads();
  if (t == 0) a.objp[I * a.NT + J] = (sm.red[0] + sm.red[1]) + (sm.red[2] + sm.red[3]);
}

template <typename T>
__global__ __launch_bounds__(NT) void k_stage(StageArgs a) {
  __shared__ StageSmem sm;
  const int b = blockIdx.x;
  if (b < a.nsweep) {
    const int I = a.ilo + b;
    run_sweep<T>(a, I, a.stage - I, sm.s);
  } else {
    run_bin(a, a.bins[b - a.nsweep], sm.t);
  }
}

// ---------------------------------------------------------------------------
// Batched rounding: independent problems (each with its own factors, X, Z, Y
// and workspace region) share the stage launches. Launch k holds the stage-k
// work groups of every problem that has a stage k: problem p owns the blocks
// off[p] .. off[p+1]-1 and runs them exactly as k_stage would, so the merged
// launch has the work of all problems in flight at once (small problems
// occupy a few compute units each). Problem p's record in a device table
// holds what differs between calls; the rest of its StageArgs is its
// handle's, kept on the device with the handle.
constexpr int BATCH_MAX = 512;  // problems per launch (block offsets travel as kernel arguments)
struct BatchProb {
  const StageArgs* base;  // the handle's fixed part (shape, factors, plan)
  const void* X;
  int32_t* Z;
  void* Y;
  int64_t ldx, ldz, ldy, cstep;
  void* ws;  // the problem's workspace region (layout of carve_workspace)
};
struct BatchLaunch {
  const BatchProb* desc;
  int* flags;  // the batch's error word
  int count, stage;
  int off[BATCH_MAX + 1];
};

__device__ __forceinline__ StageArgs batch_args(const BatchProb& q, int* flags) {
  StageArgs a = *q.base;
  a.X = q.X;
  a.ldx = q.ldx;
  a.Z = q.Z;
  a.ldz = q.ldz;
  a.Y = q.Y;
  a.ldy = q.ldy;
  a.cstep = (int)q.cstep;
  const Workspace w = carve_workspace(q.ws, a.mp, a.np, a.MT, a.NT);
  a.objp = w.objp;
  a.P = w.P;
  a.R = w.R;
  a.E = w.E;
  a.C = w.C;
  a.flags = flags;
  return a;
}

template <typename T>
__global__ __launch_bounds__(NT) void k_stage_batch(BatchLaunch bl) {
  __shared__ StageSmem sm;
  const int b = blockIdx.x;
  // the last p with off[p] <= b (problems without a stage k own no block)
  int lo = 0, hi = bl.count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (bl.off[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  StageArgs a = batch_args(bl.desc[lo], bl.flags);
  const int k = bl.stage, lb = b - bl.off[lo];
  const int4 st = a.stab[k];
  a.stage = k;
  int ihi;
  stage_rows(a.MT, a.NT, k, a.ilo, ihi);
  a.nsweep = ihi - a.ilo + 1;
  a.tasks = a.tasks ? a.tasks + st.x : nullptr;
  a.bins = a.bins ? a.bins + st.y : nullptr;
  if (lb < a.nsweep) {
    const int I = a.ilo + lb;
    run_sweep<T>(a, I, k - I, sm.s);
  } else {
    run_bin(a, a.bins[lb - a.nsweep], sm.t);
  }
}

// Objective of every problem of a batch: block p sums problem p's per-tile
// partials in a fixed order.
__global__ __launch_bounds__(NT) void k_obj_reduce_batch(const BatchProb* desc, double* out) {
  __shared__ double red[NT];
  const BatchProb& q = desc[blockIdx.x];
  const int count = q.base->MT * q.base->NT;
  const double* objp = carve_workspace(q.ws, q.base->mp, q.base->np, q.base->MT, q.base->NT).objp;
  double s = 0.0;
  for (int i = threadIdx.x; i < count; i += NT) s += objp[i];
  red[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int i = 0; i < NT; ++i) tot += red[i];
    out[blockIdx.x] = tot;
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

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t workspace_bytes(const Factors& f) {
  const size_t tile = (size_t)f.mp * f.np * sizeof(double);
  return 256 + align256((size_t)f.MT * f.NT * sizeof(double)) + 4 * tile;
}

Workspace workspace_carve(const Factors& f, void* base) {
  return carve_workspace(base, f.mp, f.np, f.MT, f.NT);
}

// Delivery plan of the deferred feedback. Targets are grouped in 2 x 2
// super-tiles (fewer at an odd edge); for super-tile rows {2a, 2a+1} and
// columns {2b, 2b+1} the down direction gets
//   - source tile rows 0 .. 2a-4 in batches of g, as products onto the whole
//     super-tile (up to 128 x 128), each in a launch after its sources are
//     swept and at least two launches before the super-tile's first sweep;
//   - source rows 2a-3 .. 2a-2 onto rows 2a, 2a+1 of one tile column c at a
//     time, in launch 2a + c - 1 (the last before tile (2a, c) is swept);
//   - source row 2a-1 onto tile (2a+1, c), in launch 2a + c;
// (source row 2a-1 of tile (2a, c) and 2a of tile (2a+1, c) are the sweeping
// workgroup's own neighbour products). The right direction is the same with
// rows and columns exchanged. Every target gets each source once, at most one
// delivery per launch, the first one (in launch order) overwriting.
//
// The far batches have a window of launches; they are placed earliest-
// deadline-first into the room that each launch leaves beside its tile
// sweeps (a launch lasts at least one tile sweep, so deliveries that fit in
// that time on the idle compute units are free), and otherwise at their
// deadline. Batches of one super-tile and direction get distinct launches.
// Task word: x = dir | overwrite << 1 | (rows - 1) << 2 | (cols - 1) << 3
// (rows, cols in tiles), y = first target tile row, z = first target tile
// column, w = first source | (one past the last source) << 16.
void schedule_tasks(int MT, int NTt, int g, std::vector<int4>& all, std::vector<int>& off) {
  const int S = MT + NTt - 1;
  if (g < 1) g = 1;
  std::vector<std::vector<int4>> per(S);
  std::vector<double> load(S, 0.0);
  auto work = [](int nr, int nc, int k) { return (double)nr * nc * k; };  // in 64^3 units
  auto emit = [&](int launch, int dir, int ti, int tj, int nr, int nc, int s0, int s1) {
    per[launch].push_back(make_int4(dir | ((nr - 1) << 2) | ((nc - 1) << 3), ti, tj, s0 | (s1 << 16)));
    load[launch] += work(nr, nc, s1 - s0);
  };
  struct Batch {
    int release, deadline, slot, dir, r0, c0, nr, nc, s0, s1;
  };
  std::vector<Batch> batches;
  int nslot = 0;
  for (int a = 0; 2 * a < MT; ++a) {
    for (int b = 0; 2 * b < NTt; ++b) {
      const int r0 = 2 * a, c0 = 2 * b;
      const int nr = std::min(2, MT - r0), nc = std::min(2, NTt - c0);
      for (int dir = 0; dir < 2; ++dir, ++nslot) {
        // along: the target index that sources run along (rows for down)
        const int t0 = dir == 0 ? r0 : c0, nt = dir == 0 ? nr : nc;
        const int o0 = dir == 0 ? c0 : r0, no = dir == 0 ? nc : nr;  // the other index
        // far sources 0 .. t0-4, batched; batch beta of nb may go no later
        // than latest - (nb - 1 - beta), which keeps distinct launches
        // feasible (its sources are swept one launch after the previous
        // batch's at the latest)
        const int far = t0 - 4;
        const int latest = r0 + c0 - 2;  // two launches before the first sweep
        const int nbatch = far >= 0 ? far / g + 1 : 0;
        for (int beta = 0; beta < nbatch; ++beta) {
          const int s0 = beta * g, sl = std::min(far, s0 + g - 1);
          batches.push_back(Batch{sl + o0 + no, latest - (nbatch - 1 - beta), nslot, dir, r0, c0, nr, nc, s0,
                                  sl + 1});
        }
        // near sources t0-3 .. t0-2 onto both targets along, one other index at a time
        if (t0 - 2 >= 0) {
          const int s0 = std::max(0, t0 - 3);
          for (int o = o0; o < o0 + no; ++o) {
            const int launch = t0 + o - 1;
            if (dir == 0) emit(launch, 0, r0, o, nt, 1, s0, t0 - 1);
            else emit(launch, 1, o, c0, 1, nt, s0, t0 - 1);
          }
        }
        // source t0-1 onto the second target along only
        if (nt == 2 && t0 - 1 >= 0) {
          for (int o = o0; o < o0 + no; ++o) {
            const int launch = t0 + o;
            if (dir == 0) emit(launch, 0, r0 + 1, o, 1, 1, t0 - 1, t0);
            else emit(launch, 1, o, c0 + 1, 1, 1, t0 - 1, t0);
          }
        }
      }
    }
  }
  // room per launch beside its sweeps: the idle compute units for the
  // duration of one tile sweep, in 64^3-product units (about 16 per unit
  // and sweep on a 256-unit device; only the ratio between launches and the
  // total matter for the placement)
  std::vector<std::vector<int>> released(S);
  for (int i = 0; i < (int)batches.size(); ++i) released[batches[i].release].push_back(i);
  auto later = [&](int x, int y) {
    return batches[x].deadline != batches[y].deadline ? batches[x].deadline > batches[y].deadline : x > y;
  };
  std::priority_queue<int, std::vector<int>, decltype(later)> avail(later);
  std::vector<int> slot_at(nslot, -1);
  for (int k = 0; k < S; ++k) {
    for (int i : released[k]) avail.push(i);
    const int nsweep = std::min(k, MT - 1) - std::max(0, k - NTt + 1) + 1;
    const double room = 16.0 * std::max(0, 256 - nsweep);
    std::vector<int> held;
    while (!avail.empty()) {
      const int i = avail.top();
      const Batch& bt = batches[i];
      const bool due = bt.deadline <= k;
      if (!due && load[k] >= room) break;
      avail.pop();
      if (slot_at[bt.slot] == k) {  // this super-tile already has a delivery here
        held.push_back(i);
        continue;
      }
      slot_at[bt.slot] = k;
      emit(k, bt.dir, bt.r0, bt.c0, bt.nr, bt.nc, bt.s0, bt.s1);
    }
    for (int i : held) avail.push(i);
  }
  // overwrite flag: the first delivery in launch order into each target
  std::vector<char> seen((size_t)2 * MT * NTt, 0);
  all.clear();
  off.assign(S + 1, 0);
  for (int k = 0; k < S; ++k) {
    // biggest products first, so the short ones fill in behind them
    std::stable_sort(per[k].begin(), per[k].end(), [](const int4& x, const int4& y) {
      const int wx = ((x.w >> 16) - (x.w & 0xffff)) * (((x.x >> 2) & 1) + 1) * (((x.x >> 3) & 1) + 1);
      const int wy = ((y.w >> 16) - (y.w & 0xffff)) * (((y.x >> 2) & 1) + 1) * (((y.x >> 3) & 1) + 1);
      return wx > wy;
    });
    for (int4& tk : per[k]) {
      const int dir = tk.x & 1;
      char& f = seen[2 * ((size_t)tk.y * NTt + tk.z) + dir];
      if (!f) tk.x |= 2;
      const int nr = ((tk.x >> 2) & 1) + 1, nc = ((tk.x >> 3) & 1) + 1;
      for (int r = 0; r < nr; ++r)
        for (int c = 0; c < nc; ++c) seen[2 * ((size_t)(tk.y + r) * NTt + tk.z + c) + dir] = 1;
    }
    off[k] = (int)all.size();
    all.insert(all.end(), per[k].begin(), per[k].end());
  }
  off[S] = (int)all.size();
}

// Bins of a stage: one per compute unit, filled longest-processing-time
// first with an estimated cost per task (microseconds per 32-deep chunk by
// target size, plus a start cost that is larger when the old target values
// are read), so that the bins finish close together; a work group per
// non-empty bin, after the sweeps. The first units - nsweep bins start
// beside the sweeps; the others only when a sweep is done, so they start
// loaded with its duration (and stay empty when the work fits beside the
// sweeps).
// (least-squares fit of measured bin durations at 4096 and 8192)
constexpr double kSweepCost = 45.0;   // one tile sweep
constexpr double kChunk4 = 5.1;       // 32-deep chunk onto 2 x 2 tiles
constexpr double kChunk2 = 2.4;       // onto 2 x 1 or 1 x 2 tiles
constexpr double kChunk1 = 1.2;       // onto one tile
constexpr double kStartOw = 1.0;      // a delivery that overwrites
constexpr double kStartAdd = 6.0;     // a delivery that adds to the old values
gptq2d_status pack_bins(int MT, int NTt, int units, std::vector<int4>& all,
                        const std::vector<int>& off, std::vector<int4>& bins, std::vector<int>& boff) {
  const int S = MT + NTt - 1;
  bins.clear();
  boff.assign(S + 1, 0);
  std::vector<int4> out;
  out.reserve(all.size());
  auto cost = [](const int4& x) {
    const int K = (x.w >> 16) - (x.w & 0xffff);
    const int tiles = (((x.x >> 2) & 1) + 1) * (((x.x >> 3) & 1) + 1);
    const double chunk = tiles == 4 ? kChunk4 : tiles == 2 ? kChunk2 : kChunk1;
    return ((x.x >> 1) & 1 ? kStartOw : kStartAdd) + chunk * (TB / KQ) * K;
  };
  for (int k = 0; k < S; ++k) {
    boff[k] = (int)bins.size();
    const int n = off[k + 1] - off[k];
    if (n == 0) continue;
    const int nsweep = std::min(k, MT - 1) - std::max(0, k - NTt + 1) + 1;
    const int nfree = std::max(0, units - nsweep);
    const int nb = std::max(1, units);
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = off[k] + i;
    std::stable_sort(order.begin(), order.end(),
                     [&](int x, int y) { return cost(all[x]) > cost(all[y]); });
    std::vector<std::vector<int>> member(nb);
    // least-loaded bin first (ties: lowest index)
    typedef std::pair<double, int> Load;
    std::priority_queue<Load, std::vector<Load>, std::greater<Load>> heap;
    for (int b = 0; b < nb; ++b) heap.push(Load(b < nfree ? 0.0 : kSweepCost, b));
    for (int i : order) {
      Load top = heap.top();
      heap.pop();
      member[top.second].push_back(i);
      top.first += cost(all[i]);
      heap.push(top);
    }
    const int base = (int)out.size();
    for (int b = 0; b < nb; ++b) {
      if (member[b].empty()) continue;
      // grouped by target shape: 2 x 2, 2 x 1, 1 x 2, 1 x 1
      if (member[b].size() > 0xffff) {
        set_error("delivery plan: too many products in one bin");
        return GPTQ2D_ERR_INVALID_ARG;
      }
      int cnt[4] = {0, 0, 0, 0};
      const int first = (int)out.size() - base;
      for (int g = 0; g < 4; ++g)
        for (int i : member[b]) {
          const int nr = ((all[i].x >> 2) & 1) + 1, nc = ((all[i].x >> 3) & 1) + 1;
          const int sh = nr == 2 ? (nc == 2 ? 0 : 1) : (nc == 2 ? 2 : 3);
          if (sh == g) out.push_back(all[i]), ++cnt[g];
        }
      bins.push_back(make_int4(first, cnt[0] | (cnt[1] << 16), cnt[2] | (cnt[3] << 16), 0));
    }
  }
  boff[S] = (int)bins.size();
  all.swap(out);
  return GPTQ2D_OK;
}

void free_schedule(Schedule& sc) {
  if (sc.d_tasks) (void)hipFree(sc.d_tasks);
  if (sc.d_bins) (void)hipFree(sc.d_bins);
  if (sc.d_stage) (void)hipFree(sc.d_stage);
  if (sc.d_base) (void)hipFree(sc.d_base);
  sc.d_tasks = nullptr;
  sc.d_bins = nullptr;
  sc.d_stage = nullptr;
  sc.d_base = nullptr;
}

gptq2d_status build_schedule(Factors& f, int g) {
  std::vector<int4> all;
  std::vector<int> off;
  if (g < 1) g = 1;
  schedule_tasks(f.MT, f.NT, g, all, off);
  int units = 0;
  if (hipDeviceGetAttribute(&units, hipDeviceAttributeMultiprocessorCount, f.device) != hipSuccess ||
      units <= 0)
    units = 256;
  std::vector<int4> bins;
  std::vector<int> boff;
  const gptq2d_status st = pack_bins(f.MT, f.NT, units, all, off, bins, boff);
  if (st != GPTQ2D_OK) return st;
  free_schedule(f.sched);
  if (!all.empty()) {
    hipError_t e = hipMalloc(&f.sched.d_tasks, all.size() * sizeof(int4));
    if (e != hipSuccess) return hip_fail(e, "schedule allocation");
    e = hipMemcpy(f.sched.d_tasks, all.data(), all.size() * sizeof(int4), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "schedule upload");
    e = hipMalloc(&f.sched.d_bins, bins.size() * sizeof(int4));
    if (e != hipSuccess) return hip_fail(e, "schedule allocation");
    e = hipMemcpy(f.sched.d_bins, bins.data(), bins.size() * sizeof(int4), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "schedule upload");
  }
  {
    const int S = f.MT + f.NT - 1;
    std::vector<int4> stab(S);
    for (int k = 0; k < S; ++k) stab[k] = int4{off[k], boff[k], boff[k + 1] - boff[k], 0};
    hipError_t e = hipMalloc(&f.sched.d_stage, S * sizeof(int4));
    if (e != hipSuccess) return hip_fail(e, "schedule allocation");
    e = hipMemcpy(f.sched.d_stage, stab.data(), S * sizeof(int4), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "schedule upload");
    // the fixed stage arguments of the handle (batched rounding)
    StageArgs b{};
    b.m = f.m;
    b.n = f.n;
    b.mp = f.mp;
    b.np = f.np;
    b.MT = f.MT;
    b.NT = f.NT;
    b.L = f.L;
    b.U = f.U;
    b.dL = f.dL;
    b.dU = f.dU;
    b.tasks = f.sched.d_tasks;
    b.bins = f.sched.d_bins;
    b.stab = f.sched.d_stage;
    e = hipMalloc(&f.sched.d_base, sizeof(StageArgs));
    if (e != hipSuccess) return hip_fail(e, "schedule allocation");
    e = hipMemcpy(f.sched.d_base, &b, sizeof(StageArgs), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "schedule upload");
  }
  f.sched.g = g;
  f.sched.stages = f.MT + f.NT - 1;
  f.sched.offset = off;
  f.sched.bin_offset = boff;
  f.sched.ntasks = all.size();
  return GPTQ2D_OK;
}

template <typename T>
static StageArgs stage_args(const Factors& f, const void* X, int64_t ldx, int32_t* Z, int64_t ldz,
                            void* Y, int64_t ldy, const Workspace& ws) {
  StageArgs a{};
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
  if (f.rev) {  // the index-reversed problem: X[m-1-i][n-1-j] etc.
    const int64_t last_x = (int64_t)(f.m - 1) * ldx + (f.n - 1);
    const int64_t last_z = (int64_t)(f.m - 1) * ldz + (f.n - 1);
    const int64_t last_y = (int64_t)(f.m - 1) * ldy + (f.n - 1);
    a.X = (const T*)X + last_x;
    a.ldx = -ldx;
    a.Z = Z + last_z;
    a.ldz = -ldz;
    a.Y = Y ? (void*)((T*)Y + last_y) : nullptr;
    a.ldy = -ldy;
    a.cstep = -1;
  } else {
    a.X = X;
    a.ldx = ldx;
    a.Z = Z;
    a.ldz = ldz;
    a.Y = Y;
    a.ldy = ldy;
    a.cstep = 1;
  }
  a.P = ws.P;
  a.R = ws.R;
  a.E = ws.E;
  a.C = ws.C;
  a.objp = ws.objp;
  a.flags = ws.flags;
  return a;
}

// work groups of stage k of a problem: the tile sweeps beside the delivery bins
static int stage_blocks(const Factors& f, int k) {
  int ilo, ihi;
  stage_rows(f.MT, f.NT, k, ilo, ihi);
  return (ihi - ilo + 1) + (f.sched.bin_offset[k + 1] - f.sched.bin_offset[k]);
}

template <typename T>
static gptq2d_status round_typed(const Factors& f, const void* X, int64_t ldx, int32_t* Z,
                                 int64_t ldz, void* Y, int64_t ldy, double* objective,
                                 const Workspace& ws, hipStream_t s, bool allow_timing) {
  StageArgs a = stage_args<T>(f, X, ldx, Z, ldz, Y, ldy, ws);
  hipLaunchKernelGGL(k_zero_flags, dim3(1), dim3(64), 0, s, ws.flags);
  const Schedule& S = f.sched;
  for (int k = 0; k < S.stages; ++k) {
    int ilo, ihi;
    stage_rows(f.MT, f.NT, k, ilo, ihi);
    a.stage = k;
    a.ilo = ilo;
    a.nsweep = ihi - ilo + 1;
    const int ntasks = S.bin_offset[k + 1] - S.bin_offset[k];  // work groups beside the sweeps
    a.tasks = S.d_tasks ? S.d_tasks + S.offset[k] : nullptr;
    a.bins = S.d_bins ? S.d_bins + S.bin_offset[k] : nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (f.stage_timing && allow_timing) {
      while (f.stage_ev.size() < f.stage_ev_used + 2) {
        hipEvent_t ev;
        hipError_t e = hipEventCreate(&ev);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
        f.stage_ev.push_back(ev);
      }
      e0 = f.stage_ev[f.stage_ev_used];
      e1 = f.stage_ev[f.stage_ev_used + 1];
      f.stage_ev_used += 2;
    }
    // with timing on, the two events take the start and end time stamps of
    // the dispatch itself (no marker packets between the launches)
    hipExtLaunchKernelGGL(k_stage<T>, dim3(a.nsweep + ntasks), dim3(NT), 0, s, e0, e1, 0, a);
  }
  if (objective)
    hipLaunchKernelGGL(k_obj_reduce, dim3(1), dim3(NT), 0, s, ws.objp, f.MT * f.NT, objective);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "sweep launch");
  return GPTQ2D_OK;
}

gptq2d_status launch_round(const Factors& f, gptq2d_dtype dt, const void* X, int64_t ldx,
                           int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                           const Workspace& ws, hipStream_t s, bool allow_timing) {
  if (dt == GPTQ2D_F32) return round_typed<float>(f, X, ldx, Z, ldz, Y, ldy, objective, ws, s, allow_timing);
  return round_typed<double>(f, X, ldx, Z, ldz, Y, ldy, objective, ws, s, allow_timing);
}

// Workspace of a batch: the batch's error flags (256 bytes), the problems'
// StageArgs table, then one gptq2d_round workspace region per problem.
static size_t batch_table_bytes(int count) { return align256((size_t)count * sizeof(BatchProb)); }

size_t batched_workspace_bytes(int count, const Factors* const* f) {
  size_t b = 256 + batch_table_bytes(count);
  for (int p = 0; p < count; ++p) b += align256(workspace_bytes(*f[p]));
  return b;
}

template <typename T>
static gptq2d_status round_batched_typed(int count, const Factors* const* f, const void* const* X,
                                         const int64_t* ldx, int32_t* const* Z, const int64_t* ldz,
                                         void* const* Y, const int64_t* ldy, double* objective,
                                         void* workspace, hipStream_t s) {
  static_assert(sizeof(BatchProb) % sizeof(uint64_t) == 0, "the table is uploaded in 8-byte words");
  char* base = (char*)workspace;
  int* flags = (int*)base;
  BatchProb* desc = (BatchProb*)(base + 256);
  char* region = base + 256 + batch_table_bytes(count);
  std::vector<BatchProb> h(count);
  for (int p = 0; p < count; ++p) {
    const Workspace ws = workspace_carve(*f[p], region);
    // X, Z, Y as the problem's sweep addresses them (mirrored in reverse order)
    const StageArgs a = stage_args<T>(*f[p], X[p], ldx[p], Z[p], ldz[p], Y ? Y[p] : nullptr, Y ? ldy[p] : 0, ws);
    h[p] = BatchProb{(const StageArgs*)f[p]->sched.d_base, a.X, a.Z, a.Y, a.ldx, a.ldz, a.ldy, a.cstep, region};
    region += align256(workspace_bytes(*f[p]));
  }
  hipLaunchKernelGGL(k_zero_flags, dim3(1), dim3(64), 0, s, flags);
  const gptq2d_status st = enqueue_upload(desc, h.data(), h.size() * sizeof(BatchProb), s);
  if (st != GPTQ2D_OK) return st;
  for (int g0 = 0; g0 < count; g0 += BATCH_MAX) {
    const int cnt = std::min(BATCH_MAX, count - g0);
    int smax = 0;
    for (int q = 0; q < cnt; ++q) smax = std::max(smax, f[g0 + q]->sched.stages);
    BatchLaunch bl;
    bl.desc = desc + g0;
    bl.flags = flags;
    bl.count = cnt;
    for (int k = 0; k < smax; ++k) {
      int tot = 0;
      for (int q = 0; q < cnt; ++q) {
        bl.off[q] = tot;
        if (k < f[g0 + q]->sched.stages) tot += stage_blocks(*f[g0 + q], k);
      }
      bl.off[cnt] = tot;
      bl.stage = k;
      hipLaunchKernelGGL(k_stage_batch<T>, dim3(tot), dim3(NT), 0, s, bl);
    }
  }
  if (objective) hipLaunchKernelGGL(k_obj_reduce_batch, dim3(count), dim3(NT), 0, s, desc, objective);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "batched sweep launch");
  return GPTQ2D_OK;
}

gptq2d_status launch_round_batched(int count, const Factors* const* f, gptq2d_dtype dt,
                                   const void* const* X, const int64_t* ldx, int32_t* const* Z,
                                   const int64_t* ldz, void* const* Y, const int64_t* ldy,
                                   double* objective, void* workspace, hipStream_t s) {
  if (dt == GPTQ2D_F32)
    return round_batched_typed<float>(count, f, X, ldx, Z, ldz, Y, ldy, objective, workspace, s);
  return round_batched_typed<double>(count, f, X, ldx, Z, ldz, Y, ldy, objective, workspace, s);
}

}  // namespace g2d
