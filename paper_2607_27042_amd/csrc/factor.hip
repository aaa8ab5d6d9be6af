// Feedback factors of the two-sided metric on the GPU.
//
// For a Gram matrix Q (G = A^T A for the rows, H = B B^T for the columns,
// Eq. GH) the rounding feedback is the unit-lower LDL factor F of Q^{-1}
// (Sec. 3.1), and U = F(H)^T (Sec. 4.1). Instead of inverting Q and factoring
// the inverse, this file uses an equivalent route that needs only a Cholesky
// factorisation and one triangular inverse:
//   Q = R R^T with R upper  =>  Q^{-1} = R^{-T} R^{-1} = F diag(R)^{-2} F^T,
//   F = R^{-T} diag(R)  (unit lower),  Lambda = diag(R)^{-2}.
// R is obtained from the ordinary lower Cholesky factor Lc of the index-
// reversed Gram J Q J (J the reversal permutation): R = J Lc J. Hence, with
// Li = Lc^{-1},
//   F[i][j] = Li[d-1-j][d-1-i] * Lc[d-1-j][d-1-j]   (i > j),
//   1 / Lambda[i] = Lc[d-1-i][d-1-i]^2.
// All work is fp64 on 64 x 64 tiles: the Gram (a SYRK), a right-looking
// blocked Cholesky (diagonal block in LDS, panel solve and trailing update on
// MFMA) and a right-looking blocked triangular inverse (MFMA).
#include <math.h>

#include <algorithm>
#include <cstring>
#include <type_traits>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace g2d {

// One side of the factorisation (0: rows, Gram G = A^T A; 1: columns,
// Gram H = B B^T), all fp64, padded to dp = nb * 64.
struct Side {
  double* gr;    // reversed Gram; its lower tiles become the Cholesky factor Lc
  double* li;    // Lc^{-1} (lower tiles)
  double* dinv;  // inverses of the 64 x 64 diagonal blocks of Lc (nb x 64 x 64)
  double* out;   // the feedback factor: L (side 0) or U (side 1)
  double* dout;  // 1 / Lambda
  int d, dp, nb;
};

struct FacArgs {
  Side s[2];
  int* flags;
  int* genv;  // Gram envelopes and work plan (GramView)
  int rev;    // reverse order: the index-reversed problem (A P, P B), so no reversal below
};

// Batched factorisation: problems of one shape in common launches. Problem p
// owns the blocks p per .. p per + per - 1 of a launch (per = the grid of a
// single problem's launch) and takes its inputs from a device table, its
// FacArgs from its handle's copy on the device; every block then does exactly
// what it does in a single problem's launch, so the results are the same bits.
struct FacStatic {  // fixed per handle
  FacArgs f;        // (f.rev unused: the order is the problem's)
  double* gpart;
};
struct FacProb {
  const FacStatic* base;
  const void* A;
  const void* B;
  int64_t lda, ldb, rev;
};
struct BatchCtx {
  const FacProb* tab;  // unused by single-problem launches
  int per;
};
template <bool BAT>
__device__ __forceinline__ const FacProb* bat_prob(const BatchCtx& bc) {
  return BAT ? bc.tab + blockIdx.x / bc.per : nullptr;
}
template <bool BAT>
__device__ __forceinline__ int bat_block(const BatchCtx& bc) {
  return BAT ? (int)(blockIdx.x % bc.per) : (int)blockIdx.x;
}
template <bool BAT>
__device__ __forceinline__ int bat_grid(const BatchCtx& bc) {
  return BAT ? bc.per : (int)gridDim.x;
}

// Lower-triangle enumeration of tile pairs: b -> (i, j) with i >= j.
__device__ __forceinline__ void tri_index(int b, int& i, int& j) {
  int r = (int)((sqrt(8.0 * (double)b + 1.0) - 1.0) * 0.5);
  while (r * (r + 1) / 2 > b) --r;
  while ((r + 1) * (r + 2) / 2 <= b) ++r;
  i = r;
  j = b - r * (r + 1) / 2;
}

// left operand given k-major in registers, r[s] = A[i][k] at k = e >> 6, i = e & 63
__device__ __forceinline__ void put_ak(Stage64& st, const double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    st.a[e >> 6][e & 63] = r[s];
  }
}

// acc += A (64 x 64) * op(B) (64 x 64) for one 64-deep block; A row-major at
// pa; B row-major at pb (BT = 0) or given as B^T row-major (BT = 1).
template <int BT>
__device__ __forceinline__ void gemm64(Acc& acc, const double* pa, int64_t lda, const double* pb,
                                       int64_t ldb, Stage64& st) {
  double ra[16], rb[16];
  load_blk(pa, lda, ra);
  load_blk(pb, ldb, rb);
  put_a(st, ra);
  if (BT) put_bt(st, rb);
  else put_b(st, rb);
  __syncthreads();
  mma_blk(acc, st);
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Reversed Gram Gr[p][q] = sum_k S(k, p) S(k, q) with the index reversal
// folded into the loads: S(k, p) = A[k][d-1-p] (side 0), B[d-1-p][k] (side 1).
// Lower tiles of both sides in one grid; identity block on the padding.
// ---------------------------------------------------------------------------

template <typename T, int SIDE>
__device__ __forceinline__ void gram_load(const T* S, int64_t ld, int d, int i0, int k0, double r[16],
                                          int rev) {
  const int t = threadIdx.x;
  T v[16];
  bool ok[16];
  // unconditional loads from clamped addresses (no per-load branch), then
  // zero what lies outside the matrix
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s, hi = e >> 6, lo = e & 63;
    int64_t off;
    // (in reverse order the problem is (A P, P B): A[k][idx], B[idx][k])
    if (SIDE == 0) {  // (k = hi, i = lo): A[k0+k][d-1-(i0+i)], coalesced along i
      const int k = k0 + hi, idx = i0 + lo;
      ok[s] = k < d && idx < d;
      off = (int64_t)k * ld + (rev ? idx : d - 1 - idx);
    } else {          // (i = hi, k = lo): B[d-1-(i0+i)][k0+k], coalesced along k
      const int idx = i0 + hi, k = k0 + lo;
      ok[s] = k < d && idx < d;
      off = (int64_t)(rev ? idx : d - 1 - idx) * ld + k;
    }
    v[s] = S[ok[s] ? off : 0];
  }
#pragma unroll
  for (int s = 0; s < 16; ++s) r[s] = ok[s] ? (double)v[s] : 0.0;
}

template <typename T, int SIDE>
__device__ void gram_tile(const Side& sd, const T* S, int64_t ld, int bp, int bq, Stage64& st, int rev) {
  Acc acc;
  acc.zero();
  double ra[16], rb[16];
  gram_load<T, SIDE>(S, ld, sd.d, bp * TB, 0, ra, rev);
  gram_load<T, SIDE>(S, ld, sd.d, bq * TB, 0, rb, rev);
  const int nk = (sd.d + TB - 1) / TB;
  for (int kb = 0; kb < nk; ++kb) {
    if (SIDE == 0) {
      put_ak(st, ra);
      put_b(st, rb);
    } else {
      put_a(st, ra);
      put_bt(st, rb);
    }
    __syncthreads();
    if (kb + 1 < nk) {  // next block's loads in flight during this block's MFMAs
      gram_load<T, SIDE>(S, ld, sd.d, bp * TB, (kb + 1) * TB, ra, rev);
      gram_load<T, SIDE>(S, ld, sd.d, bq * TB, (kb + 1) * TB, rb, rev);
    }
    mma_blk(acc, st);
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int pp = bp * TB + acc_row(u, r), qq = bq * TB + acc_col(v);
        double val = acc.t[2 * u + v][r];
        if (pp >= sd.d || qq >= sd.d) val = (pp == qq) ? 1.0 : 0.0;
        sd.gr[(int64_t)pp * sd.dp + qq] = val;
      }
}

// Sides in a Gram launch: side 0 if bit 0 of `sides` is set, side 1 if bit
// 1 is; the grid holds the lower tiles of the first, then of the second.
template <typename T, bool BAT>
__global__ __launch_bounds__(NT) void k_gram(FacArgs f0, const T* A0, int64_t lda0, const T* B0,
                                             int64_t ldb0, int sides, BatchCtx bc) {
  __shared__ Stage64 st;
  const FacProb* pb = bat_prob<BAT>(bc);
  const FacArgs& f = BAT ? pb->base->f : f0;
  const T* A = BAT ? (const T*)pb->A : A0;
  const T* B = BAT ? (const T*)pb->B : B0;
  const int64_t lda = BAT ? pb->lda : lda0, ldb = BAT ? pb->ldb : ldb0;
  const int bid = bat_block<BAT>(bc);
  const int rev = BAT ? (int)pb->rev : f0.rev;
  const int t0 = (sides & 1) ? f.s[0].nb * (f.s[0].nb + 1) / 2 : 0;
  int bp, bq;
  if (bid < t0) {
    tri_index(bid, bp, bq);
    gram_tile<T, 0>(f.s[0], A, lda, bp, bq, st, rev);
  } else {
    tri_index(bid - t0, bp, bq);
    gram_tile<T, 1>(f.s[1], B, ldb, bp, bq, st, rev);
  }
}

// ---------------------------------------------------------------------------
// Gram of a side whose dimension is a multiple of 128, in two steps.
//
// k_gram_prep writes, widened to fp64, the row-major panel S (d x d, row
// stride d) whose rows are the reversed Gram indices: S[p][k] = A[k][d-1-p]
// (side 0, a transpose through LDS) or B[d-1-p][k] (side 1); in reverse order
// the problem is already the index-reversed one, S[p][k] = A[k][p] or B[p][k].
// The panel lives in the side's inverse buffer, which the factorisation fills
// only later.
//
// While it writes the panel, k_gram_prep also records each 128-row block's
// envelope: the range of 64-column blocks holding a nonzero entry. Entry
// (p, q) of the Gram only gathers products S[p][k] S[q][k] with k in both
// rows' envelopes; every other term is an exact zero, and adding it leaves a
// floating-point sum unchanged, so the contraction of tile (bp, bq) runs over
// the intersection of the two row blocks' envelopes and gives the same Gram.
// A triangular basis (the Cholesky factor of a Gram, as in every workload
// here) leaves about a third of the dense contraction; a dense one all of it.
// k_gram_plan turns the envelopes into each tile's range of 32-deep chunks
// and the division of all of them between the work groups (below).
//
// k_gram128 then forms Gr[p][q] = sum_k S[p][k] S[q][k] on the lower
// 128 x 128 tiles: four waves, each a 64 x 64 quadrant as 4 x 4 MFMA blocks
// (the upper quadrant of a diagonal tile is computed but not stored), the
// 32-deep chunks of both 128-row panels streamed by direct global -> LDS
// loads into double buffers (the same layout as the delivery products: row
// blocks of four, 16-byte pieces XOR-permuted by the row's position in the
// block, 64 bytes of padding per block).
// ---------------------------------------------------------------------------

// The chunks of all 128 x 128 Gram tiles, tile by tile (side 0's tiles
// first), form one sequence of work units, dealt out as G contiguous ranges
// of nearly equal length, one per work group, so that no round of work groups
// runs with most of the device idle. A range is at least as long as the
// longest tile: a tile is either inside one range (stored directly) or split
// between two neighbouring ranges, whose partial products go to a pair of
// scratch slots (one per range boundary) and are added by k_gram_fix in a
// fixed order. A tile's chunks are those its envelope leaves (an empty
// intersection counts as one unit that stores zeros), so the division is
// made on the device by k_gram_plan; the host fixes the launch grid from the
// dense count, an upper bound for G.
struct GramPlan {
  int t0, t1;          // tiles of side 0 and side 1 on this path
  int n0, n1;          // 128-row blocks of side 0 and side 1 on this path
  int nch0, nch1;      // dense chunks per tile on each side
  int64_t units;       // dense units: t0 nch0 + t1 nch1
  int G;               // launch grid (work groups, an upper bound for the ranges)
};

// The envelope and plan buffer of a handle (ints): the total of units (an
// int64) and the number of ranges, each tile's first and one past its last
// chunk, the prefix sum of the tiles' unit counts (int64), and per side the
// nonzero votes of the panel's 64 x 64 blocks (one int per wave of the prep
// kernel's work group: (d/64)^2 x 4).
struct GramView {
  long long* U;
  int* Geff;
  int* clo;
  int* chi;
  long long* pre;
  int* mask[2];
};
// (offsets in ints from a 256-byte aligned base: pre on 8 bytes, the votes
// on 16 bytes, read as int4)
__host__ __device__ inline size_t gram_pre_at(int T) { return (4 + 2 * (size_t)T + 1) / 2 * 2; }
__host__ __device__ inline size_t gram_mask_at(int T) { return (gram_pre_at(T) + 2 * ((size_t)T + 1) + 3) / 4 * 4; }
__host__ __device__ inline size_t gram_view_ints(int n0, int n1, int T) {
  return gram_mask_at(T) + 16 * (size_t)n0 * n0 + 16 * (size_t)n1 * n1;
}
__host__ __device__ inline GramView gram_view(int* base, int n0, int n1, int T) {
  GramView v;
  v.U = (long long*)base;
  v.Geff = base + 2;
  v.clo = base + 4;
  v.chi = v.clo + T;
  v.pre = (long long*)(base + gram_pre_at(T));
  v.mask[0] = base + gram_mask_at(T);
  v.mask[1] = v.mask[0] + 16 * (size_t)n0 * n0;
  return v;
}
__device__ __forceinline__ GramView gram_view(int* base, const GramPlan& pl) {
  return gram_view(base, pl.n0, pl.n1, pl.t0 + pl.t1);
}

// Unit u (0 <= u < U) -> its tile: the last t with pre[t] <= u.
__device__ __forceinline__ int gram_tile_of(const long long* pre, int T, long long u) {
  int lo = 0, hi = T - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= u) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

constexpr int GQ = 32;           // chunk depth
constexpr int GA = 4 * GQ + 8;   // doubles per 4-row block
struct GramChunk {
  double a[32][GA];   // rows 128 bp ..
  double b[32][GA];   // rows 128 bq ..
};

template <typename T, bool BAT>
__global__ __launch_bounds__(NT) void k_gram_prep(FacArgs f0, const T* A0, int64_t lda0, const T* B0,
                                                  int64_t ldb0, int sides, GramPlan pl, BatchCtx bc) {
  __shared__ double tile[TB][TB + 1];
  const FacProb* pb = bat_prob<BAT>(bc);
  const FacArgs& f = BAT ? pb->base->f : f0;
  const T* A = BAT ? (const T*)pb->A : A0;
  const T* B = BAT ? (const T*)pb->B : B0;
  const int64_t lda = BAT ? pb->lda : lda0, ldb = BAT ? pb->ldb : ldb0;
  const int n0 = (sides & 1) ? (f.s[0].d / TB) * (f.s[0].d / TB) : 0;
  int b = bat_block<BAT>(bc);
  const int side = b < n0 ? 0 : 1;
  if (side == 1) b -= n0;
  const Side& sd = f.s[side];
  const int d = sd.d, nt = d / TB;
  const int i0 = (b / nt) * TB, k0 = (b % nt) * TB;  // S rows i0.., columns k0..
  double* S = sd.li;
  const int t = threadIdx.x;
  const int rev = BAT ? (int)pb->rev : f0.rev;
  bool nz = false;  // a nonzero entry in this thread's part of the block
  if (side == 0) {
    // A rows k0 + r, columns d-1-(i0+63) .. d-1-i0 (ascending; in reverse
    // order i0 .. i0+63), coalesced
    const int c0 = rev ? i0 : d - i0 - TB;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = t + NT * u, r = e >> 6, c = e & 63;  // c: column offset in A
      const double x = (double)A[(int64_t)(k0 + r) * lda + c0 + c];
      tile[r][c] = x;
      nz |= x != 0.0;
    }
    __syncthreads();
    // S[i0 + i][k0 + k] = A[k0 + k][d-1-(i0+i)] = tile[k][63 - i] (reverse order: tile[k][i])
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = t + NT * u, i = e >> 6, k = e & 63;
      S[(int64_t)(i0 + i) * d + k0 + k] = tile[k][rev ? i : TB - 1 - i];
    }
  } else {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = t + NT * u, i = e >> 6, k = e & 63;
      const int row = rev ? i0 + i : d - 1 - (i0 + i);
      const double x = (double)B[(int64_t)row * ldb + k0 + k];
      S[(int64_t)(i0 + i) * d + k0 + k] = x;
      nz |= x != 0.0;
    }
  }
  // each wave's vote whether its part of the block holds a nonzero entry
  // (a NaN counts as nonzero); k_gram_plan turns the votes into envelopes
  const int any = __any(nz) ? 1 : 0;
  if ((threadIdx.x & 63) == 0) {
    const GramView v = gram_view(f.genv, pl);
    v.mask[side][((int64_t)(i0 >> 6) * nt + (k0 >> 6)) * 4 + (threadIdx.x >> 6)] = any;
  }
}

// (i0, i1 select the part i0 <= i < i1 of the loads)
__device__ __forceinline__ void gram_issue(const double* Sp, const double* Sq, int64_t ld, int c,
                                           GramChunk& g, int w, int l, int i0 = 0, int i1 = 8) {
  typedef __attribute__((address_space(3))) void lds_v;
  const int ar = l >> 4, ap = (l & 15) ^ ar;
  const int64_t k0 = (int64_t)c * GQ + 2 * ap;
#pragma unroll
  for (int i = i0; i < i1; ++i) {
    const int j = w + 4 * i;
    const int64_t ro = (int64_t)(4 * j + ar) * ld + k0;
    __builtin_amdgcn_global_load_lds((const void*)(Sp + ro), (lds_v*)&g.a[j][0], 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)(Sq + ro), (lds_v*)&g.b[j][0], 16, 0, 0);
  }
}

// Every tile's chunk range from the envelopes of its two row blocks, the
// prefix sum of the unit counts, and the number of ranges: the launch grid,
// or fewer so that a range is at least as long as the longest tile.
constexpr int PLT = 1024;
constexpr int PLE = 512;  // 128-row blocks per side (dimensions up to 65536)
template <bool BAT>
__global__ __launch_bounds__(PLT) void k_gram_plan(FacArgs f0, GramPlan pl, BatchCtx bc) {
  __shared__ long long scan[2][PLT];
  __shared__ int mx[PLT];
  __shared__ int env[2][2][PLE];  // [side][first, one past last][128-row block]
  const FacProb* pb = bat_prob<BAT>(bc);
  const FacArgs& f = BAT ? pb->base->f : f0;
  const GramView v = gram_view(f.genv, pl);
  const int T = pl.t0 + pl.t1, t = threadIdx.x;
  // envelopes of the 128-row blocks from the votes of the panel's 64 x 64
  // blocks (start empty: first past last)
  for (int i = t; i < 2 * PLE; i += PLT) {
    env[i / PLE][0][i % PLE] = 0x7fffffff;
    env[i / PLE][1][i % PLE] = 0;
  }
  __syncthreads();
  for (int side = 0; side < 2; ++side) {
    const int nk = 2 * (side ? pl.n1 : pl.n0);  // 64 x 64 blocks per panel row and column
    const int4* votes = (const int4*)v.mask[side];
    for (int e = t; e < nk * nk; e += PLT) {
      const int4 q = votes[e];
      if (q.x | q.y | q.z | q.w) {
        atomicMin(&env[side][0][(e / nk) >> 1], e % nk);
        atomicMax(&env[side][1][(e / nk) >> 1], e % nk + 1);
      }
    }
  }
  __syncthreads();
  auto emin = [&](int side, int b) { return env[side][0][b]; };
  auto emax = [&](int side, int b) { return env[side][1][b]; };
  const int per = (T + PLT - 1) / PLT, a0 = min(T, t * per), a1 = min(T, a0 + per);
  long long sum = 0;
  int most = 0;
  for (int i = a0; i < a1; ++i) {
    const int side = i < pl.t0 ? 0 : 1;
    int bp, bq;
    tri_index(side ? i - pl.t0 : i, bp, bq);
    const int lo = max(emin(side, bp), emin(side, bq)), hi = min(emax(side, bp), emax(side, bq));
    const bool empty = hi <= lo;
    v.clo[i] = empty ? 0 : 2 * lo;  // an envelope block is two 32-deep chunks
    v.chi[i] = empty ? 0 : 2 * hi;
    const int cnt = empty ? 1 : 2 * (hi - lo);
    sum += cnt;
    most = max(most, cnt);
  }
  // inclusive scan of the threads' sums (Hillis-Steele) and the largest tile
  scan[0][t] = sum;
  mx[t] = most;
  __syncthreads();
  int cur = 0;
  for (int off = 1; off < PLT; off <<= 1) {
    const long long x = scan[cur][t] + (t >= off ? scan[cur][t - off] : 0);
    const int y = t + off < PLT ? max(mx[t], mx[t + off]) : mx[t];
    __syncthreads();
    scan[cur ^ 1][t] = x;
    mx[t] = y;  // mx[0] ends as the maximum
    cur ^= 1;
    __syncthreads();
  }
  const long long total = scan[cur][PLT - 1];
  if (t == 0) {
    *v.U = total;
    *v.Geff = (int)max(1LL, min((long long)pl.G, total / max(mx[0], 1)));
    v.pre[T] = total;
  }
  long long run = scan[cur][t] - sum;  // exclusive
  for (int i = a0; i < a1; ++i) {
    v.pre[i] = run;
    run += v.chi[i] > v.clo[i] ? v.chi[i] - v.clo[i] : 1;
  }
}

// Chunks c0 .. c1-1 of the tile (bp, bq) of one side into acc (zeroed here).
__device__ __forceinline__ void gram_part(const Side& sd, int bp, int bq, int c0, int c1, GramChunk* buf,
                                          d4 (&acc)[4][4]) {
  const int d = sd.d;
  const double* Sp = sd.li + (int64_t)(128 * bp) * d;
  const double* Sq = sd.li + (int64_t)(128 * bq) * d;
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  const int qr = w >> 1, qc = w & 1, r0 = l & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};
  if (c0 < c1) gram_issue(Sp, Sq, d, c0, buf[0], w, l);
  for (int c = c0; c < c1; ++c) {
    const int cb = (c - c0) & 1;
    // the next chunk's loads in two halves, the second half-way through this
    // chunk's MFMAs (one batch stalls the wave's issue until the memory
    // pipeline takes it)
    const bool more = c + 1 < c1;
    if (more) {
      gram_issue(Sp, Sq, d, c + 1, buf[cb ^ 1], w, l, 0, 4);
      __builtin_amdgcn_s_waitcnt(0x0f78);  // vmcnt(8): chunk c has landed
    } else {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    }
    asm volatile("s_barrier" ::: "memory");  // the wait above covers this wave's part
    const GramChunk& st = buf[cb];
    // operands of k-step kk + 1 are read while kk is on MFMA (two register
    // sets), the reads spread between the MFMAs
    double av[2][4], bv[2][4];
    const int rr = r0 & 3;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ao = GQ * rr + 2 * ((l >> 5) ^ rr) + ((l >> 4) & 1);
      av[0][i] = st.a[(64 * qr + 16 * i + r0) >> 2][ao];
      bv[0][i] = st.b[(64 * qc + 16 * i + r0) >> 2][ao];
    }
#pragma unroll
    for (int kk = 0; kk < GQ / 4; ++kk) {
      const int cur = kk & 1, nx = cur ^ 1;
      if (kk == GQ / 8 && more) {
        __builtin_amdgcn_sched_barrier(0);
        gram_issue(Sp, Sq, d, c + 1, buf[cb ^ 1], w, l, 4, 8);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (kk + 1 < GQ / 4) {
        const int kp = 2 * (kk + 1) + (l >> 5), ao = GQ * rr + 2 * (kp ^ rr) + ((l >> 4) & 1);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          av[nx][i] = st.a[(64 * qr + 16 * i + r0) >> 2][ao];
          bv[nx][i] = st.b[(64 * qc + 16 * i + r0) >> 2][ao];
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[cur][i], bv[cur][j], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two MFMAs
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // buffer refilled next
  }
}

// The wave's 64 x 64 quadrant of a finished tile into the Gram (the upper
// quadrant of a diagonal tile is not kept).
__device__ __forceinline__ void gram_store(const Side& sd, int bp, int bq, const d4 (&acc)[4][4]) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, qr = w >> 1, qc = w & 1;
  if (bp == bq && qr < qc) return;
  double* o = sd.gr + (int64_t)(128 * bp + 64 * qr + (l >> 4)) * sd.dp + 128 * bq + 64 * qc + (l & 15);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[(int64_t)(16 * i + 4 * r) * sd.dp + 16 * j] = acc[i][j][r];
}

// Scratch slot of a partial product: every thread keeps its 64 values in
// the accumulator order, 256 threads side by side.
__device__ __forceinline__ double* gram_slot(double* part, int slot, int h) {
  return part + ((int64_t)(2 * slot + h) << 14) + threadIdx.x;
}

template <bool BAT>
__global__ __launch_bounds__(NT) void k_gram128(FacArgs f0, GramPlan pl, double* part0, BatchCtx bc) {
  __shared__ GramChunk buf[2];
  const FacProb* pb = bat_prob<BAT>(bc);
  const FacArgs& f = BAT ? pb->base->f : f0;
  double* part = BAT ? pb->base->gpart : part0;
  const GramView v = gram_view(f.genv, pl);
  const int bid = bat_block<BAT>(bc);
  const int G = *v.Geff, T = pl.t0 + pl.t1;
  const long long U = *v.U;
  // work groups are dealt round-robin to the eight L2 domains (XCDs): give
  // each domain a contiguous run of ranges, so that the tiles it runs at the
  // same time share their row panel (tri_index enumerates row by row)
  // (domain x holds the work groups i = x mod 8 and gets q ranges, plus one
  // when x < r, from x q + min(x, r) on, with q, r the quotient and remainder
  // of G by 8; the launch's further work groups have none)
  const int q8 = G / 8, r8 = G % 8;
  const int x = bid % 8, y = bid / 8;
  if (y >= q8 + (x < r8 ? 1 : 0)) return;
  const int jr = x * q8 + min(x, r8) + y;
  const long long lo = U * jr / G, hi = U * (jr + 1) / G;
  d4 acc[4][4];
  int tile = lo < hi ? gram_tile_of(v.pre, T, lo) : 0;
  for (long long u = lo; u < hi; ++tile) {
    const int side = tile < pl.t0 ? 0 : 1;
    const Side& sd = f.s[side];
    const long long p0 = v.pre[tile], p1 = v.pre[tile + 1];
    const int clo = v.clo[tile], nreal = v.chi[tile] - clo;
    const int o0 = (int)(u - p0), o1 = (int)(min(p1, hi) - p0);  // this range's units of the tile
    const int c0 = clo + min(o0, nreal), c1 = clo + min(o1, nreal);
    int bp, bq;
    tri_index(side ? tile - pl.t0 : tile, bp, bq);
    if (u != lo) __syncthreads();  // the staging buffers are reused
    gram_part(sd, bp, bq, c0, c1, buf, acc);
    if (u == p0 && min(p1, hi) == p1) {
      gram_store(sd, bp, bq, acc);
    } else {
      // the head of a tile ends this range (slot jr), the tail of one starts it (slot jr - 1)
      double* o = u == p0 ? gram_slot(part, jr, 0) : gram_slot(part, jr - 1, 1);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[(int64_t)(((i * 4 + j) * 4 + r) * NT)] = acc[i][j][r];
    }
    u = min(p1, hi);
  }
}

// Tiles split between ranges jr and jr + 1: head + tail, stored as a finished tile.
template <bool BAT>
__global__ __launch_bounds__(NT) void k_gram_fix(FacArgs f0, GramPlan pl, const double* part0, BatchCtx bc) {
  const FacProb* pb = bat_prob<BAT>(bc);
  const FacArgs& f = BAT ? pb->base->f : f0;
  const double* part = BAT ? pb->base->gpart : part0;
  const GramView v = gram_view(f.genv, pl);
  const int jr = bat_block<BAT>(bc);
  const int G = *v.Geff, T = pl.t0 + pl.t1;
  if (jr + 1 >= G) return;
  const long long u = *v.U * (jr + 1) / G;
  const int tile = gram_tile_of(v.pre, T, u);
  if (u == v.pre[tile]) return;  // the boundary falls between tiles
  const double* h0 = gram_slot(const_cast<double*>(part), jr, 0);
  const double* h1 = gram_slot(const_cast<double*>(part), jr, 1);
  d4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t e = (int64_t)(((i * 4 + j) * 4 + r) * NT);
        acc[i][j][r] = h0[e] + h1[e];
      }
  const int side = tile < pl.t0 ? 0 : 1;
  int bp, bq;
  tri_index(side ? tile - pl.t0 : tile, bp, bq);
  gram_store(f.s[side], bp, bq, acc);
}

static GramPlan gram_plan(int m, int n, int fast, int cus) {
  GramPlan pl;
  const int n0 = m / 128, n1 = n / 128;
  pl.n0 = (fast & 1) ? n0 : 0;
  pl.n1 = (fast & 2) ? n1 : 0;
  pl.t0 = pl.n0 * (pl.n0 + 1) / 2;
  pl.t1 = pl.n1 * (pl.n1 + 1) / 2;
  pl.nch0 = std::max(1, m / GQ);
  pl.nch1 = std::max(1, n / GQ);
  pl.units = (int64_t)pl.t0 * pl.nch0 + (int64_t)pl.t1 * pl.nch1;
  const int64_t nmax = std::max(pl.t0 ? pl.nch0 : 1, pl.t1 ? pl.nch1 : 1);
  // every range at least one dense tile long: a tile meets at most one boundary
  pl.G = (int)std::max<int64_t>(1, std::min<int64_t>(std::max(cus, 1), pl.units / nmax));
  return pl;
}

static int fast_sides(int m, int n) { return (m % 128 == 0 ? 1 : 0) | (n % 128 == 0 ? 2 : 0); }

size_t gram_part_doubles(int m, int n, int cus) {
  const int fast = fast_sides(m, n);
  if (!fast) return 0;
  const GramPlan pl = gram_plan(m, n, fast, cus);
  return pl.G > 1 ? (size_t)2 * pl.G * 16384 : 0;
}

size_t gram_env_ints(int m, int n) {
  const int fast = fast_sides(m, n);
  if (!fast) return 0;
  const GramPlan pl = gram_plan(m, n, fast, 1);
  return gram_view_ints(pl.n0, pl.n1, pl.t0 + pl.t1);
}

// ---------------------------------------------------------------------------
// Cholesky of one 64 x 64 diagonal block (already updated by all earlier
// panels) and the inverse of its lower factor; one workgroup per side.
//
// Blocked over 16 x 16 sub-blocks held in LDS. For each diagonal sub-block k:
// one wave factors it and inverts the factor in registers (16 pivots, each
// broadcast by DPP); the other sub-blocks of column k are solved against that
// inverse and the trailing sub-blocks updated, both as 16 x 16 MFMA products.
// The wave that owns the next diagonal sub-block updates it from its own
// panel first and factors it while the other waves finish their trailing
// updates, so only one panel product and one update lie between two
// factorisations. The inverse of the whole factor is assembled block row by
// block row, each row as soon as its diagonal block is inverted, by the waves
// left idle:
//   W_ij = -W_ii (sum_{k=j}^{i-1} L_ik W_kj).
// A pivot that is not positive and finite raises FLAG_SINGULAR and is
// replaced by 1 so the remaining work stays finite.
// ---------------------------------------------------------------------------

constexpr int DS = 16;  // sub-block edge

__device__ __forceinline__ double readlane_d(double v, int lane) {
  const long long x = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)x, lane);
  const int hi = __builtin_amdgcn_readlane((int)(x >> 32), lane);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// 1 / sqrt(x) for x > 0: hardware estimate and one Newton step.
__device__ __forceinline__ double rsqrt_nr(double x) {
  const double y = __builtin_amdgcn_rsq(x);
  const double h = 0.5 * x;
  return y * fma(-h * y, y, 1.5);
}

// acc += s * X (16 x K) op(Y) on MFMA; X and Y in LDS, row-major with strides
// ldx, ldy; op(Y) = Y^T with Y given as 16 x K (T = 1) or Y itself, K x 16
// (T = 0). One wave; every operand load is issued before the first MFMA.
template <int K, int T>
__device__ __forceinline__ void mfma_lds(d4& acc, const double* X, int ldx, const double* Y, int ldy,
                                         double sgn) {
  const int l = threadIdx.x & 63;
  const double* qx = X + (l & 15) * ldx + (l >> 4);
  double xv[K / 4], yv[K / 4];
#pragma unroll
  for (int s = 0; s < K / 4; ++s) {
    xv[s] = sgn * qx[4 * s];
    yv[s] = T ? Y[(l & 15) * ldy + (l >> 4) + 4 * s] : Y[((l >> 4) + 4 * s) * ldy + (l & 15)];
  }
#pragma unroll
  for (int s = 0; s < K / 4; ++s) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(xv[s], yv[s], acc, 0, 0, 0);
}

// MFMA-layout accumulator <-> a 16 x 16 LDS block (element r of lane l is
// entry (4r + l/16, l%16)).
__device__ __forceinline__ void d4_load(d4& acc, const double* P, int ld) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] = P[(4 * r + (l >> 4)) * ld + (l & 15)];
}
__device__ __forceinline__ void d4_store(const d4& acc, double* P, int ld) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int r = 0; r < 4; ++r) P[(4 * r + (l >> 4)) * ld + (l & 15)] = acc[r];
}

// v of lane `lane` (0..15, a constant after unrolling) of every 16-lane row,
// broadcast to the whole row (DPP row_newbcast, one 64-bit move).
__device__ __forceinline__ double bcast16(double v, int lane) {
  switch (lane) {
#define G2D_BC(L_) \
  case L_:         \
    return __builtin_amdgcn_mov_dpp(v, 0x150 + (L_), 0xf, 0xf, false);
    G2D_BC(0) G2D_BC(1) G2D_BC(2) G2D_BC(3) G2D_BC(4) G2D_BC(5) G2D_BC(6) G2D_BC(7)
    G2D_BC(8) G2D_BC(9) G2D_BC(10) G2D_BC(11) G2D_BC(12) G2D_BC(13) G2D_BC(14) G2D_BC(15)
#undef G2D_BC
    default: return v;
  }
}

// Factor the 16 x 16 diagonal sub-block at A (stride lda, lower part valid)
// in place and write its inverse to W (stride ldw). One wave; lane x of
// every 16-lane row holds column x of the symmetric block and column x of
// the inverse in registers, and every broadcast is a DPP broadcast of one
// lane within the row. Pivot j, with s = 1 / sqrt(S[j][j]):
//   - lane x's entry j becomes L[x][j] = S[x][j] s (x >= j), and entry j of
//     its column of the inverse is divided by L[j][j];
//   - every lane subtracts L[r][j] L[x][j] = S[r][j] (S[x][j] s^2) from its
//     entries r > j (right-looking Cholesky; entries r > x of lane x are
//     never used again), with S[r][j] broadcast from lane j, and advances the
//     column-oriented forward substitution of L W = I by the same column;
//   - entry j + 1 goes first, so that the next pivot's square root can be
//     scheduled between the remaining updates, whose broadcasts are all
//     issued before their multiply-adds.
// At the end lane x holds row x of L (entries 0..x) and column x of W.
__device__ void chol_inv16(double* A, int lda, double* W, int ldw, int* flags) {
  int l = threadIdx.x & 63;
  // opaque to the optimiser: keeps the per-lane set-up inside the caller's
  // loop instead of hoisting it out and holding it in registers throughout
  asm volatile("" : "+v"(l));
  const int x = l & 15;
  double a[DS], w[DS];
#pragma unroll
  for (int r = 0; r < DS; ++r) {
    a[r] = (r >= x) ? A[r * lda + x] : A[x * lda + r];
    w[r] = (r == x) ? 1.0 : 0.0;
  }
  __builtin_amdgcn_wave_barrier();
  bool bad = false;
  auto pivot_rs = [&](double piv) {
    const bool ok = piv > 0.0 && isfinite(piv);
    bad |= !ok;
    return rsqrt_nr(ok ? piv : 1.0);
  };
  double rs = pivot_rs(bcast16(a[0], 0));
#pragma unroll
  for (int j = 0; j < DS; ++j) {
    const double rs2 = rs * rs;
    const double c = -a[j] * rs2, cw = -w[j] * rs2;
    a[j] *= rs;
    w[j] *= rs;
    double rs_next = 1.0;
    if (j + 1 < DS) {
      const double b = bcast16(a[j + 1], j);
      a[j + 1] = fma(b, c, a[j + 1]);
      w[j + 1] = fma(b, cw, w[j + 1]);
      rs_next = pivot_rs(bcast16(a[j + 1], j + 1));
    }
    double bb[DS];
#pragma unroll
    for (int r = j + 2; r < DS; ++r) bb[r] = bcast16(a[r], j);
#pragma unroll
    for (int r = j + 2; r < DS; ++r) {
      a[r] = fma(bb[r], c, a[r]);
      w[r] = fma(bb[r], cw, w[r]);
    }
    // an empty asm keeps the pivot's updates of the inverse inside the
    // pivot: left free, the compiler defers them past the loop and parks the
    // broadcasts in spare registers, one more move per entry
    asm volatile("" : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(w[4]), "+v"(w[5]), "+v"(w[6]),
                 "+v"(w[7]), "+v"(w[8]), "+v"(w[9]), "+v"(w[10]), "+v"(w[11]), "+v"(w[12]), "+v"(w[13]),
                 "+v"(w[14]), "+v"(w[15]));
    rs = rs_next;
  }
  if (bad && l == 0) raise_flag(flags, FLAG_SINGULAR);
  // after pivot j, a[j] of lane x is L[x][j] (x >= j): each lane holds row x of
  // the factor and column x of its inverse
  if (l < DS) {
#pragma unroll
    for (int r = 0; r < DS; ++r) {
      A[x * lda + r] = (r <= x) ? a[r] : 0.0;
      W[r * ldw + x] = (r >= x) ? w[r] : 0.0;
    }
  }
}

constexpr int DLD = TB + 1;
struct DiagSmem {
  double Am[TB][DLD];      // the block, becomes Lc (lower)
  double Wm[TB][DLD];      // Lc^{-1} (lower)
  double Tm[4][DS][DS + 1];
};

// Diagonal block kb of one side by one work group: Cholesky factor in place
// (gr) and its inverse into dinv.
__device__ void diag_tile(const Side& sd, int kb, int* flags, DiagSmem& ds) {
  constexpr int LD = DLD;
  double(*Am)[LD] = ds.Am;
  double(*Wm)[LD] = ds.Wm;
  double(*Tm)[DS][DS + 1] = ds.Tm;
  const int t = threadIdx.x, w = t >> 6;
  double* blk = sd.gr + (int64_t)kb * TB * sd.dp + (int64_t)kb * TB;
  {
    double x[16];
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int e = t + NT * s;
      x[s] = blk[(int64_t)(e >> 6) * sd.dp + (e & 63)];
    }
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int e = t + NT * s, r = e >> 6, c = e & 63;
      Am[r][c] = (c <= r) ? x[s] : 0.0;
      Wm[r][c] = 0.0;
    }
  }
  __syncthreads();
  // off-diagonal block row i of the inverse, block (i, w) by wave w < i:
  // W_iw = -W_ii (sum_{m=w}^{i-1} L_im W_mw)
  auto wrow = [&](int i) {
    d4 acc = {0.0, 0.0, 0.0, 0.0};
    for (int m = w; m < i; ++m) mfma_lds<DS, 0>(acc, &Am[DS * i][DS * m], LD, &Wm[DS * m][DS * w], LD, 1.0);
    d4_store(acc, &Tm[w][0][0], DS + 1);
    __builtin_amdgcn_wave_barrier();
    d4 acc2 = {0.0, 0.0, 0.0, 0.0};
    mfma_lds<DS, 0>(acc2, &Wm[DS * i][DS * i], LD, &Tm[w][0][0], DS + 1, -1.0);
    d4_store(acc2, &Wm[DS * i][DS * w], LD);
  };
  if (w == 0) chol_inv16(&Am[0][0], LD, &Wm[0][0], LD, flags);
  __syncthreads();
  for (int k = 0; k < 3; ++k) {
    const int o = DS * k;
    if (w > k) {  // panel: L_wk = A_wk W_kk^T
      d4 acc = {0.0, 0.0, 0.0, 0.0};
      mfma_lds<DS, 1>(acc, &Am[DS * w][o], LD, &Wm[o][o], LD, 1.0);
      __builtin_amdgcn_wave_barrier();
      d4_store(acc, &Am[DS * w][o], LD);
    }
    if (w == k + 1) {  // the next diagonal block, from the wave's own panel: A_ww -= L_wk L_wk^T
      __builtin_amdgcn_wave_barrier();
      d4 acc;
      d4_load(acc, &Am[DS * w][DS * w], LD);
      mfma_lds<DS, 1>(acc, &Am[DS * w][o], LD, &Am[DS * w][o], LD, -1.0);
      d4_store(acc, &Am[DS * w][DS * w], LD);
    }
    __syncthreads();
    if (w == k + 1) {
      chol_inv16(&Am[DS * w][DS * w], LD, &Wm[DS * w][DS * w], LD, flags);
    } else if (w > k + 1) {  // trailing: A_wj -= L_wk L_jk^T, k < j <= w
      for (int j = k + 1; j <= w; ++j) {
        d4 acc;
        d4_load(acc, &Am[DS * w][DS * j], LD);
        mfma_lds<DS, 1>(acc, &Am[DS * w][o], LD, &Am[DS * j][o], LD, -1.0);
        d4_store(acc, &Am[DS * w][DS * j], LD);
      }
    } else if (w < k) {  // block row k of the inverse (W_kk is ready)
      wrow(k);
    }
    __syncthreads();
  }
  if (w < 3) wrow(3);
  __syncthreads();
  double* dv = sd.dinv + (int64_t)kb * TB * TB;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s, r = e >> 6, c = e & 63;
    blk[(int64_t)r * sd.dp + c] = Am[r][c];
    dv[e] = Wm[r][c];
  }
}

template <bool BAT>
__global__ __launch_bounds__(NT) void k_diag(FacArgs f0, int kb, BatchCtx bc) {
  __shared__ DiagSmem ds;
  const FacArgs& f = BAT ? bat_prob<BAT>(bc)->base->f : f0;
  const Side sd = f.s[bat_block<BAT>(bc)];  // a copy: the stores below cannot alias it
  int* const flags = f.flags;
  if (kb >= sd.nb) return;
  diag_tile(sd, kb, flags, ds);
}

// ---------------------------------------------------------------------------
// Panel step kb, both sides in one grid:
//   solve:  Lc[ib][kb] = Q[ib][kb] dinv[kb]^T                (ib > kb)
//   invert: Li[kb][kb] = dinv[kb];
//           Li[kb][jb] = -dinv[kb] S[kb][jb], S accumulated in place (jb < kb)
// ---------------------------------------------------------------------------

__device__ __forceinline__ int panel_count(const Side& sd, int kb) {
  return kb < sd.nb ? (sd.nb - kb - 1) + (kb + 1) : 0;
}

template <bool BAT>
__global__ __launch_bounds__(NT) void k_panel(FacArgs f0, int kb, BatchCtx bc) {
  __shared__ Stage64 st;
  const FacArgs& f = BAT ? bat_prob<BAT>(bc)->base->f : f0;
  int b = bat_block<BAT>(bc);
  const int n0 = panel_count(f.s[0], kb);
  const Side& sd = (b < n0) ? f.s[0] : f.s[1];
  if (b >= n0) b -= n0;
  const int rest = sd.nb - kb - 1;
  const double* dk = sd.dinv + (int64_t)kb * TB * TB;
  Acc acc;
  acc.zero();
  if (b < rest) {
    const int ib = kb + 1 + b;
    double* blk = sd.gr + (int64_t)ib * TB * sd.dp + (int64_t)kb * TB;
    gemm64<1>(acc, blk, sd.dp, dk, TB, st);
    acc_store(acc, blk, sd.dp, 1.0);
  } else {
    const int jb = b - rest;
    double* out = sd.li + (int64_t)kb * TB * sd.dp + (int64_t)jb * TB;
    if (jb == kb) {
      for (int e = threadIdx.x; e < TB * TB; e += NT) out[(int64_t)(e >> 6) * sd.dp + (e & 63)] = dk[e];
    } else {
      gemm64<0>(acc, dk, TB, out, sd.dp, st);
      acc_store(acc, out, sd.dp, -1.0);
    }
  }
}

// ---------------------------------------------------------------------------
// Update with the finished panels k0 .. k1-1 (both sides in one grid):
//   Q[bi][bj] -= sum_kb Lc[bi][kb] Lc[bj][kb]^T      (qa <= bj < qb, bj <= bi)
//   S[ib][jb] += sum_kb Lc[ib][kb] Li[kb][jb]        (sa <= ib < sb, jb < k1,
//                                                      max(k0, jb) <= kb < k1)
// S is the running sum of the triangular inverse, kept in place in Li; its
// first contribution (kb = jb) overwrites. Called, before each panel of a
// group, for that panel's column and row with the group's earlier panels,
// and with the whole group for everything beyond it, so the bulk of the
// trailing work is done with products as deep as the group.
// ---------------------------------------------------------------------------

struct UpdRange {
  int qa, qb, sa, sb, k0, k1;
  int j0;  // S columns from j0 on (jb in [j0, k1))
  int dg;  // the diagonal block whose update completes here (qa), factored
           // by the same work group right after it; -1: none
};

__device__ __forceinline__ void upd_counts(const Side& sd, const UpdRange& r, int& nq, int& ns) {
  nq = ns = 0;
  if (r.k0 >= sd.nb) return;
  for (int bj = r.qa; bj < min(r.qb, sd.nb); ++bj) nq += sd.nb - bj;
  ns = max(0, min(r.sb, sd.nb) - r.sa) * max(0, min(r.k1, sd.nb) - r.j0);
}

// acc += sum over 64-deep blocks b of A_b op(B_b), A_b at pa + b*sa_, B_b at
// pb + b*sb_; BT: B given transposed. Double-buffered through LDS.
template <int BT>
__device__ void gemm_blocks(Acc& acc, const double* pa, int64_t lda, int64_t sa_, const double* pb,
                            int64_t ldb, int64_t sb_, int nb, Stage64* st) {
  double ra[16], rb[16];
  load_blk(pa, lda, ra);
  load_blk(pb, ldb, rb);
  for (int b = 0; b < nb; ++b) {
    Stage64& s = st[b & 1];
    put_a(s, ra);
    if (BT) put_bt(s, rb);
    else put_b(s, rb);
    __syncthreads();
    if (b + 1 < nb) {
      load_blk(pa + (b + 1) * sa_, lda, ra);
      load_blk(pb + (b + 1) * sb_, ldb, rb);
    }
    mma_blk(acc, s);
  }
}

template <bool BAT>
__global__ __launch_bounds__(NT) void k_update(FacArgs f0, UpdRange r, BatchCtx bc) {
  __shared__ union {
    Stage64 st[2];
    DiagSmem d;
  } sm;
  Stage64* st = sm.st;
  const FacArgs& f = BAT ? bat_prob<BAT>(bc)->base->f : f0;
  int b = bat_block<BAT>(bc);
  int nq0, ns0;
  upd_counts(f.s[0], r, nq0, ns0);
  // the two sides' diagonal blocks (the first Q tile of each side) go to
  // the first two work groups: their factorisation is the longest chain
  if (r.dg >= 0 && nq0 + ns0 > 1 && nq0 + ns0 < bat_grid<BAT>(bc)) {
    if (b == 1) b = nq0 + ns0;
    else if (b == nq0 + ns0) b = 1;
  }
  const bool s1 = b >= nq0 + ns0;
  const Side sd = s1 ? f.s[1] : f.s[0];  // a copy: the stores below cannot alias it
  if (s1) b -= nq0 + ns0;
  int nq, ns;
  upd_counts(sd, r, nq, ns);
  const int k1 = min(r.k1, sd.nb);
  Acc acc;
  acc.zero();
  if (b < nq) {
    int bj = r.qa;
    while (b >= sd.nb - bj) {
      b -= sd.nb - bj;
      ++bj;
    }
    const int bi = bj + b;
    gemm_blocks<1>(acc, sd.gr + (int64_t)bi * TB * sd.dp + (int64_t)r.k0 * TB, sd.dp, TB,
                   sd.gr + (int64_t)bj * TB * sd.dp + (int64_t)r.k0 * TB, sd.dp, TB, k1 - r.k0, st);
    double* out = sd.gr + (int64_t)bi * TB * sd.dp + (int64_t)bj * TB;
    double old[2][2][4];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int q = 0; q < 4; ++q) old[u][v][q] = out[(int64_t)acc_row(u, q) * sd.dp + acc_col(v)];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          out[(int64_t)acc_row(u, q) * sd.dp + acc_col(v)] = old[u][v][q] - acc.t[2 * u + v][q];
    if (bi == r.dg && bj == r.dg) {
      // no other work group of this launch reads this block (their operands
      // are columns before k1 <= dg); its factorisation starts as soon as it
      // is complete (written above, read back by the same work group)
      __syncthreads();
      diag_tile(sd, r.dg, f.flags, sm.d);
    }
  } else {
    b -= nq;
    const int ib = r.sa + b / (k1 - r.j0), jb = r.j0 + b % (k1 - r.j0);
    const int kb0 = max(r.k0, jb);
    double* out = sd.li + (int64_t)ib * TB * sd.dp + (int64_t)jb * TB;
    if (jb < r.k0) acc_add_from(acc, out, sd.dp);
    gemm_blocks<0>(acc, sd.gr + (int64_t)ib * TB * sd.dp + (int64_t)kb0 * TB, sd.dp, TB,
                   sd.li + (int64_t)kb0 * TB * sd.dp + (int64_t)jb * TB, sd.dp, (int64_t)TB * sd.dp,
                   k1 - kb0, st);
    acc_store(acc, out, sd.dp, 1.0);
  }
}

// ---------------------------------------------------------------------------
// The far part of a group's trailing update on 128 x 128 tiles, for the
// group of panels g0 .. g1-1 and the block columns of Q / block rows of S
// g2 .. g3-1 (g0, g2 even; g3 even or at least the block count, which
// means up to the end):
//   Q tiles (BI >= BJ, g2/2 <= BJ < g3/2):  Q -= Lc[BI][g0:g1] Lc[BJ][g0:g1]^T
//   S tiles (g2/2 <= BI < g3/2, BJ < g0/2): S += Lc[BI][g0:g1] Li[g0:g1][BJ]
// with the same meaning as in k_update (the group's own S columns stay
// there). Four waves, each a 64 x 64 quadrant as 4 x 4 MFMA blocks; the
// accumulators start from the old values (the left operand enters negated
// for Q); 32-deep chunks of both operands by direct global -> LDS loads,
// double-buffered, in the layouts of the Gram tiles (rows with a contiguous
// contraction index) and, for the right operand of S, rows of Li (b[k][j]).
// A tile past the last block row / column (odd block count) is loaded from
// clamped rows and its missing quadrants are not stored.
// ---------------------------------------------------------------------------

struct UpdChunk {
  double a[32][GA];
  union {
    double bt[32][GA];         // right operand given as rows (Q)
    double b[GQ][2 * TB + 2];  // right operand rows k (S)
  };
};

// Work groups of the far update: eight waves, two per SIMD, so that one
// wave's MFMAs run while the other waits (load issue, barrier).
constexpr int UT = 512;

// Chunk c of both operands into d: the 32 four-row blocks of each, wave w
// the blocks j = w + 8 i (i0 <= i < i1 of i < 4).
template <int BT>
__device__ __forceinline__ void upd_issue(const double* Ap, int64_t lda, const double* Bp, int64_t ldb,
                                          int c, int nr, int nc, UpdChunk& d, int w, int l, int i0 = 0,
                                          int i1 = 4) {
  typedef __attribute__((address_space(3))) void lds_v;
  const int ar = l >> 4, ap = (l & 15) ^ ar;
  const int64_t k0 = (int64_t)c * GQ;
#pragma unroll
  for (int i = i0; i < i1; ++i) {
    const int j = w + 8 * i;
    const double* pa = Ap + (int64_t)min(4 * j + ar, TB * nr - 1) * lda + k0 + 2 * ap;
    __builtin_amdgcn_global_load_lds((const void*)pa, (lds_v*)&d.a[j][0], 16, 0, 0);
    if (BT) {
      const double* pb = Bp + (int64_t)min(4 * j + ar, TB * nc - 1) * ldb + k0 + 2 * ap;
      __builtin_amdgcn_global_load_lds((const void*)pb, (lds_v*)&d.bt[j][0], 16, 0, 0);
    } else {
      const double* pb = Bp + (k0 + j) * ldb + min(2 * l, TB * nc - 2);
      __builtin_amdgcn_global_load_lds((const void*)pb, (lds_v*)&d.b[j][0], 16, 0, 0);
    }
  }
}

// One 128 x 128 tile: wave w computes rows 64 qr .., columns 64 qc + 32 h ..
// (qr = (w >> 1) & 1, qc = w & 1, h = w >> 2) as 4 x 2 MFMA blocks.
template <int BT>
__device__ void upd_tile(double* out, int64_t ldo, const double* Ap, int64_t lda, const double* Bp,
                         int64_t ldb, int K, int nr, int nc, bool diag, UpdChunk* buf) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  const int qr = (w >> 1) & 1, qc = w & 1, h = w >> 2, r0 = l & 15, rr = r0 & 3;
  const bool mine = qr < nr && qc < nc && !(diag && qr < qc);
  const double sgn = BT ? -1.0 : 1.0;
  const int cb = 64 * qc + 32 * h;
  double* o = out + (int64_t)(64 * qr + (l >> 4)) * ldo + cb + (l & 15);
  d4 acc[4][2];
  upd_issue<BT>(Ap, lda, Bp, ldb, 0, nr, nc, buf[0], w, l);
  if (mine) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] = o[(int64_t)(16 * i + 4 * r) * ldo + 16 * j];
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): no wait for them inside the loop
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};
  }
  const int nch = K / GQ;
  for (int c = 0; c < nch; ++c) {
    // the next chunk's loads in two halves, the second half-way through this
    // chunk's MFMAs
    const bool more = c + 1 < nch;
    if (more) {
      upd_issue<BT>(Ap, lda, Bp, ldb, c + 1, nr, nc, buf[(c + 1) & 1], w, l, 0, 2);
      __builtin_amdgcn_s_waitcnt(0x0f74);  // vmcnt(4): chunk c has landed
    } else {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    }
    asm volatile("s_barrier" ::: "memory");  // the wait above covers this wave's part
    const UpdChunk& st = buf[c & 1];
    double av[2][4], bv[2][2];
#pragma unroll
    for (int kk = -1; kk < GQ / 4; ++kk) {
      const int nx = (kk + 1) & 1;
      if (kk == GQ / 8 && more) {
        __builtin_amdgcn_sched_barrier(0);
        upd_issue<BT>(Ap, lda, Bp, ldb, c + 1, nr, nc, buf[(c + 1) & 1], w, l, 2, 4);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (kk + 1 < GQ / 4) {
        const int k = 4 * (kk + 1) + (l >> 4), kp = 2 * (kk + 1) + (l >> 5);
        const int ao = GQ * rr + 2 * (kp ^ rr) + ((l >> 4) & 1);
#pragma unroll
        for (int i = 0; i < 4; ++i) av[nx][i] = sgn * st.a[(64 * qr + 16 * i + r0) >> 2][ao];
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bv[nx][j] = BT ? st.bt[(cb + 16 * j + r0) >> 2][ao] : st.b[k][cb + 16 * j + r0];
      }
      if (kk >= 0) {
        const int cur = kk & 1;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[cur][i], bv[cur][j], acc[i][j], 0, 0, 0);
        if (kk + 1 < GQ / 4) {
#pragma unroll
          for (int u = 0; u < 6; ++u) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // buffer refilled next
  }
  if (mine) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[(int64_t)(16 * i + 4 * r) * ldo + 16 * j] = acc[i][j][r];
  }
}

// Q tiles in the 128-wide block columns t0 <= BJ < t1 (every row BI >= BJ)
// and S tiles in the block rows t0 <= BI < t1; t1 = nb2 is the whole
// trailing triangle, enumerated row by row, a narrower range column by column.
__host__ __device__ __forceinline__ int far_q_count(int nb2, int t0, int t1) {
  return t1 >= nb2 ? (nb2 - t0) * (nb2 - t0 + 1) / 2 : (t1 - t0) * (2 * nb2 - t0 - t1 + 1) / 2;
}

__device__ void update128_tile(const FacArgs& f, int g0, int g1, int g2, int g3, int b, UpdChunk* buf) {
  for (int s = 0; s < 2; ++s) {
    const Side& sd = f.s[s];
    const int nb = sd.nb;
    if (g0 >= nb || g1 <= g0) continue;
    const int nb2 = (nb + 1) / 2, t0 = g2 / 2, t1 = g3 >= nb ? nb2 : g3 / 2;
    if (t0 >= t1) continue;
    const int nq = far_q_count(nb2, t0, t1), ns = (t1 - t0) * (g0 / 2);
    const int K = TB * (min(g1, nb) - g0);
    const int64_t dp = sd.dp;
    if (b < nq) {
      int BI, BJ;
      if (t1 >= nb2) {
        int bi, bj;
        tri_index(b, bi, bj);  // bi >= bj, relative to t0
        BI = t0 + bi;
        BJ = t0 + bj;
      } else {
        BJ = t0;
        while (b >= nb2 - BJ) {
          b -= nb2 - BJ;
          ++BJ;
        }
        BI = BJ + b;
      }
      upd_tile<1>(sd.gr + (int64_t)128 * BI * dp + 128 * BJ, dp,
                  sd.gr + (int64_t)128 * BI * dp + TB * g0, dp,
                  sd.gr + (int64_t)128 * BJ * dp + TB * g0, dp, K,
                  min(2, nb - 2 * BI), min(2, nb - 2 * BJ), BI == BJ, buf);
      return;
    }
    b -= nq;
    if (b < ns) {
      const int BI = t0 + b / (g0 / 2), BJ = b % (g0 / 2);
      upd_tile<0>(sd.li + (int64_t)128 * BI * dp + 128 * BJ, dp,
                  sd.gr + (int64_t)128 * BI * dp + TB * g0, dp,
                  sd.li + (int64_t)TB * g0 * dp + 128 * BJ, dp, K,
                  min(2, nb - 2 * BI), 2, false, buf);
      return;
    }
    b -= ns;
  }
}

// ntile tiles over the grid, tile b by work group b mod gridDim.x: a grid
// smaller than the device leaves compute units to the diagonal blocks and
// panels that run beside it on the other stream
template <bool BAT>
__global__ __launch_bounds__(UT) void k_update128(FacArgs f0, int g0, int g1, int g2, int g3, int ntile,
                                                  BatchCtx bc) {
  __shared__ UpdChunk buf[2];
  const FacArgs& f = BAT ? bat_prob<BAT>(bc)->base->f : f0;
  const int bid = bat_block<BAT>(bc), grid = bat_grid<BAT>(bc);
  // work groups are dealt round-robin to the eight L2 domains: each domain
  // takes a contiguous run of every round's tiles, so that the tiles it runs
  // at the same time share their row panel (rows are enumerated tile by tile)
  const int q8 = grid / 8, r8 = grid % 8, x = bid % 8;
  const int pos = x * q8 + min(x, r8) + bid / 8;
  for (int b = pos; b < ntile; b += grid) {
    if (b != pos) __syncthreads();  // the staging buffers are reused
    update128_tile(f, g0, g1, g2, g3, b, buf);
  }
}

// ---------------------------------------------------------------------------
// Normalisation into the feedback factor and 1/Lambda (both sides):
//   side 0: L[i][j] = Li[d-1-j][d-1-i] Lc[d-1-j][d-1-j]  (i > j), lower tiles
//   side 1: U[i][j] = Li[d-1-i][d-1-j] Lc[d-1-i][d-1-i]  (j > i), upper tiles
//   1/Lambda[i] = Lc[d-1-i][d-1-i]^2; the padding becomes an identity block.
// L is stored tile by tile in S order, U in R order (device.hpp); only the
// triangle's tiles are written, and only they are ever read.
// ---------------------------------------------------------------------------

template <bool BAT>
__global__ __launch_bounds__(NT) void k_finalize(FacArgs f0, BatchCtx bc) {
  __shared__ double S[TB][TB + 1];
  __shared__ double sc[TB];
  const FacArgs& f = BAT ? bat_prob<BAT>(bc)->base->f : f0;
  const int bid = bat_block<BAT>(bc);
  const int t0 = f.s[0].nb * (f.s[0].nb + 1) / 2;
  const int side = bid < t0 ? 0 : 1;
  const Side& sd = f.s[side];
  int bi, bj;
  tri_index(side == 0 ? bid : bid - t0, bi, bj);  // bi >= bj
  const int d = sd.d, dp = sd.dp;
  const int rs = d - TB - bj * TB, cs = d - TB - bi * TB;
  const int t = threadIdx.x;
  for (int e = t; e < TB * TB; e += NT) {
    const int x = e >> 6, y = e & 63, r = rs + x, c = cs + y;
    S[x][y] = (r >= 0 && r < d && c >= 0 && c < d) ? sd.li[(int64_t)r * dp + c] : 0.0;
  }
  if (t < TB) {
    const int r = rs + t;
    sc[t] = (r >= 0 && r < d) ? sd.gr[(int64_t)r * dp + r] : 1.0;
  }
  __syncthreads();
  const int orow = side == 0 ? bi : bj, ocol = side == 0 ? bj : bi;
  for (int e = t; e < TB * TB; e += NT) {
    const int a = e >> 6, b = e & 63;
    const int i = orow * TB + a, j = ocol * TB + b;
    double val;
    if (i >= d || j >= d || i == j) {
      val = (i == j) ? 1.0 : 0.0;
    } else if (side == 0) {
      val = (i > j) ? S[63 - b][63 - a] * sc[63 - b] : 0.0;
    } else {
      val = (j > i) ? S[63 - a][63 - b] * sc[63 - a] : 0.0;
    }
    sd.out[side == 0 ? s_at(i, j, sd.nb) : r_at(i, j, sd.nb)] = val;
  }
  if (bi == bj && t < TB) {
    const int i = bi * TB + t;
    sd.dout[i] = (i < d) ? sc[63 - t] * sc[63 - t] : 1.0;
  }
}

__global__ void k_zero_flags_batch(const FacProb* tab, int count) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < count) tab[p].base->f.flags[0] = 0;
}

// Stream-ordered upload of up to PUT_WORDS 8-byte words that travel as
// kernel arguments (no host buffer has to outlive the enqueueing call).
constexpr int PUT_WORDS = 384;
struct PutArgs {
  uint64_t* dst;
  int n;
  uint64_t w[PUT_WORDS];
};
__global__ void k_put(PutArgs p) {
  for (int i = threadIdx.x; i < p.n; i += blockDim.x) p.dst[i] = p.w[i];
}

static gptq2d_status check_launch(const char* what);

gptq2d_status enqueue_upload(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes % sizeof(uint64_t) != 0 || ((uintptr_t)dst) % sizeof(uint64_t) != 0) {
    set_error("upload of a partial word");
    return GPTQ2D_ERR_INVALID_ARG;
  }
  const uint64_t* words = static_cast<const uint64_t*>(src);
  const size_t nwords = bytes / sizeof(uint64_t);
  for (size_t w0 = 0; w0 < nwords; w0 += PUT_WORDS) {
    PutArgs pa;
    pa.dst = static_cast<uint64_t*>(dst) + w0;
    pa.n = (int)std::min<size_t>(PUT_WORDS, nwords - w0);
    std::memcpy(pa.w, words + w0, pa.n * sizeof(uint64_t));
    hipLaunchKernelGGL(k_put, dim3(1), dim3(NT), 0, s, pa);
  }
  return check_launch("upload");
}

__global__ void k_zero_int(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// factor export: dense triangle out of the tiled storage (L in S order, U in
// R order), lam = 1 / dl.
__global__ void k_export_tri(const double* src, int dp, int d, double* dst, int64_t ld, int lower) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)d * d) return;
  const int i = (int)(e / d), j = (int)(e % d);
  const bool keep = lower ? (j <= i) : (j >= i);
  const int64_t at = lower ? s_at(i, j, dp / TB) : r_at(i, j, dp / TB);
  dst[(int64_t)i * ld + j] = keep ? (i == j ? 1.0 : src[at]) : 0.0;
}

__global__ void k_export_lam(const double* dl, int d, double* lam) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < d) lam[i] = 1.0 / dl[i];
}

__global__ void k_import_tri(const double* src, int64_t ld, int d, int dp, double* dst, int lower) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)dp * dp) return;
  const int i = (int)(e / dp), j = (int)(e % dp);
  double v;
  if (i == j) v = 1.0;
  else if (i >= d || j >= d) v = 0.0;
  else if (lower ? (j < i) : (j > i)) v = src[(int64_t)i * ld + j];
  else v = 0.0;
  dst[lower ? s_at(i, j, dp / TB) : r_at(i, j, dp / TB)] = v;
}

__global__ void k_import_lam(const double* lam, int d, int dp, double* dl) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < dp) dl[i] = (i < d) ? 1.0 / lam[i] : 1.0;
}

static gptq2d_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, what);
  return GPTQ2D_OK;
}

static FacArgs fac_args(Factors& f) {
  FacArgs a;
  for (int s = 0; s < 2; ++s) {
    Side& sd = a.s[s];
    sd.gr = f.gram[s];
    sd.li = f.inv[s];
    sd.dinv = f.dinv[s];
    sd.out = s == 0 ? f.L : f.U;
    sd.dout = s == 0 ? f.dL : f.dU;
    sd.d = s == 0 ? f.m : f.n;
    sd.dp = s == 0 ? f.mp : f.np;
    sd.nb = sd.dp / TB;
  }
  a.flags = f.flags;
  a.genv = f.genv;
  a.rev = f.rev;
  return a;
}

static int h_panel_count(int nb, int kb) { return kb < nb ? nb : 0; }
static int h_upd_count(int nb, const UpdRange& r) {
  if (r.k0 >= nb) return 0;
  int nq = 0;
  for (int bj = r.qa; bj < std::min(r.qb, nb); ++bj) nq += nb - bj;
  return nq + std::max(0, std::min(r.sb, nb) - r.sa) * std::max(0, std::min(r.k1, nb) - r.j0);
}

// work groups of k_update128 for one side (see there)
static void h_far_counts(int nb, int g0, int g1, int g2, int g3, int& nq, int& ns) {
  nq = ns = 0;
  if (g0 >= nb || g1 <= g0) return;
  const int nb2 = (nb + 1) / 2, t0 = g2 / 2, t1 = g3 >= nb ? nb2 : g3 / 2;
  if (t0 >= t1) return;
  nq = far_q_count(nb2, t0, t1);
  ns = (t1 - t0) * (g0 / 2);
}

// The factorisation of one problem (tab == nullptr: its inputs A, B), or of
// `count` problems of f's shape whose FacArgs and inputs are in the device
// table `tab` (A, B unused); f provides the shape, the second stream and the
// events either way.
static gptq2d_status factor_impl(Factors& f, const FacProb* tab, int count, gptq2d_dtype dt,
                                 const void* A, int64_t lda, const void* B, int64_t ldb,
                                 hipStream_t s) {
  FacArgs a = fac_args(f);
  const int nb0 = a.s[0].nb, nb1 = a.s[1].nb, nbmax = nb0 > nb1 ? nb0 : nb1;
  const int tri = nb0 * (nb0 + 1) / 2 + nb1 * (nb1 + 1) / 2;
  // launch with `per` work groups per problem
  auto go = [&](int per, hipStream_t st, auto&& launch) {
    if (per <= 0) return;
    if (!tab) launch(std::false_type{}, dim3(per), BatchCtx{nullptr, 0}, st);
    else launch(std::true_type{}, dim3(per * count), BatchCtx{tab, per}, st);
  };
  if (!tab) hipLaunchKernelGGL(k_zero_int, dim3(1), dim3(64), 0, s, f.flags, 1);
  else hipLaunchKernelGGL(k_zero_flags_batch, dim3((count + 63) / 64), dim3(64), 0, s, tab, count);
  // Gram: sides whose dimension is a multiple of 128 through the prepared
  // panel and 128 x 128 tiles, the others with 64 x 64 tiles straight from
  // the input
  int fast = 0, slow = 0, nprep = 0, nslow = 0;
  for (int sd = 0; sd < 2; ++sd) {
    const int d = a.s[sd].d, nb = a.s[sd].nb;
    if (d % 128 == 0) {
      fast |= 1 << sd;
      nprep += (d / TB) * (d / TB);
    } else {
      slow |= 1 << sd;
      nslow += nb * (nb + 1) / 2;
    }
  }
  if (fast) {
    const GramPlan pl = gram_plan(f.m, f.n, fast, f.cus);
    go(nprep, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
      constexpr bool BT = decltype(bat)::value;
      if (dt == GPTQ2D_F32)
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram_prep<float, BT>), g, dim3(NT), 0, st, a,
                           (const float*)A, lda, (const float*)B, ldb, fast, pl, bc);
      else
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram_prep<double, BT>), g, dim3(NT), 0, st, a,
                           (const double*)A, lda, (const double*)B, ldb, fast, pl, bc);
    });
    go(1, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
      constexpr bool BT = decltype(bat)::value;
      hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram_plan<BT>), g, dim3(PLT), 0, st, a, pl, bc);
    });
    go(pl.G, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
      constexpr bool BT = decltype(bat)::value;
      hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram128<BT>), g, dim3(NT), 0, st, a, pl, f.gpart, bc);
    });
    go(pl.G - 1, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
      constexpr bool BT = decltype(bat)::value;
      hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram_fix<BT>), g, dim3(NT), 0, st, a, pl,
                         (const double*)f.gpart, bc);
    });
  }
  if (slow) {
    go(nslow, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
      constexpr bool BT = decltype(bat)::value;
      if (dt == GPTQ2D_F32)
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram<float, BT>), g, dim3(NT), 0, st, a, (const float*)A,
                           lda, (const float*)B, ldb, slow, bc);
      else
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_gram<double, BT>), g, dim3(NT), 0, st, a,
                           (const double*)A, lda, (const double*)B, ldb, slow, bc);
    });
  }
  auto update = [&](const UpdRange& r, hipStream_t st) {
    go(h_upd_count(nb0, r) + h_upd_count(nb1, r), st, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t q) {
      constexpr bool BT = decltype(bat)::value;
      hipLaunchKernelGGL(HIP_KERNEL_NAME(k_update<BT>), g, dim3(NT), 0, q, a, r, bc);
    });
  };
  // The trailing update with group g0 .. g1-1 of the block columns / rows
  // ga .. gb-1 on stream st: the bulk on 128 x 128 tiles, the inverse columns
  // of the group itself (variable depth, first contribution overwrites) on
  // 64 x 64.
  auto group_update = [&](int g0, int g1, int ga, int gb, hipStream_t st0) {
    int fq0, fs0, fq1, fs1;
    h_far_counts(nb0, g0, g1, ga, gb, fq0, fs0);
    h_far_counts(nb1, g0, g1, ga, gb, fq1, fs1);
    const int nfar = fq0 + fs0 + fq1 + fs1;
    if (nfar > 0) {
      int units = 256;
      (void)hipDeviceGetAttribute(&units, hipDeviceAttributeMultiprocessorCount, f.device);
      // a far update of a few tiles per compute unit leaves at least 8 units
      // to the diagonal blocks, panels and near updates beside it (measured
      // best at 4096 among 0 to 48), and spreads its tiles evenly over as few
      // work groups as the same number of rounds needs, so that the rest of
      // the device stays free; a larger one is the longer of the two streams
      // and takes every unit (a batch fills the device by itself: one tile
      // per work group)
      int grid = nfar;
      if (!tab && nfar <= 4 * units) {
        const int rounds = (nfar + units - 9) / (units - 8);
        grid = (nfar + rounds - 1) / rounds;
      }
      go(grid, st0, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
        constexpr bool BT = decltype(bat)::value;
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_update128<BT>), g, dim3(UT), 0, st, a, g0, g1, ga, gb, nfar, bc);
      });
    }
    update(UpdRange{ga, ga, ga, gb, g0, g1, g0, -1}, st0);
  };
  // Groups of GROUP panels (an even count: the far part works on pairs of
  // block columns). Inside a group, before each panel, its column of Q and
  // row of S receive the group's earlier panels (left-looking, so that the
  // critical chain has few work groups); afterwards the whole group updates
  // everything beyond it with (64 GROUP)-deep products: the next group's
  // columns on the caller's stream (they are needed first), the rest on the
  // second stream, where it overlaps the next group's panels. The second
  // stream takes the group after next first and marks its end with an event:
  // the next group's near update writes those columns and waits for that
  // part only, not for the rest behind it. Eight panels per group from 96
  // block columns on (measured faster at 8192), four below (at 4096).
  const int GROUP = nbmax > 96 ? 8 : 4;
  hipError_t he = hipSuccess;
  bool far_pending = false, far1_pending = false;
  for (int g0 = 0; g0 < nbmax; g0 += GROUP) {
    const int g1 = std::min(g0 + GROUP, nbmax), g2 = std::min(g1 + GROUP, nbmax);
    const int g3 = std::min(g2 + GROUP, nbmax);
    for (int kb = g0; kb < g1; ++kb) {
      // the diagonal block of every later panel is factored by the update
      // that completes it (the in-group update of the panel before, or the
      // group's near update for the next group's first panel)
      if (kb == 0)
        go(2, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
          constexpr bool BT = decltype(bat)::value;
          hipLaunchKernelGGL(HIP_KERNEL_NAME(k_diag<BT>), g, dim3(NT), 0, st, a, kb, bc);
        });
      go(h_panel_count(nb0, kb) + h_panel_count(nb1, kb), s,
         [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
           constexpr bool BT = decltype(bat)::value;
           hipLaunchKernelGGL(HIP_KERNEL_NAME(k_panel<BT>), g, dim3(NT), 0, st, a, kb, bc);
         });
      // left-looking inside the group: the next panel's column of Q and row
      // of S get all of the group's finished panels at once (the later
      // columns wait for their own turn)
      if (kb + 1 < g1) update(UpdRange{kb + 1, kb + 2, kb + 1, kb + 2, g0, kb + 1, 0, kb + 1}, s);
    }
    if (far1_pending) {
      // the previous group's far update of the columns g1 .. g2-1 (and,
      // earlier on the same stream, everything older that reaches them)
      he = hipStreamWaitEvent(s, f.ev_far1, 0);
      if (he != hipSuccess) return hip_fail(he, "hipStreamWaitEvent");
      far1_pending = false;
    }
    // the next group's columns (the near update, on this stream: they are
    // needed first; 64 x 64 tiles, the first diagonal block factored by the
    // work group that completes it)
    update(UpdRange{g1, g2, g1, g2, g0, g1, 0, g1}, s);
    if (g2 < nbmax) {
      he = hipEventRecord(f.ev_near, s);
      if (he == hipSuccess) he = hipStreamWaitEvent(f.aux, f.ev_near, 0);
      if (he != hipSuccess) return hip_fail(he, "event record / wait");
      group_update(g0, g1, g2, g3, f.aux);
      he = hipEventRecord(f.ev_far1, f.aux);
      if (he != hipSuccess) return hip_fail(he, "hipEventRecord");
      far1_pending = true;
      if (g3 < nbmax) group_update(g0, g1, g3, nbmax, f.aux);
      he = hipEventRecord(f.ev_far, f.aux);
      if (he != hipSuccess) return hip_fail(he, "hipEventRecord");
      far_pending = true;
    }
  }
  if (far_pending) {
    he = hipStreamWaitEvent(s, f.ev_far, 0);
    if (he != hipSuccess) return hip_fail(he, "hipStreamWaitEvent");
  }
  go(tri, s, [&](auto bat, dim3 g, BatchCtx bc, hipStream_t st) {
    constexpr bool BT = decltype(bat)::value;
    hipLaunchKernelGGL(HIP_KERNEL_NAME(k_finalize<BT>), g, dim3(NT), 0, st, a, bc);
  });
  return check_launch("factorisation launch");
}

gptq2d_status launch_factor(Factors& f, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, hipStream_t s) {
  return factor_impl(f, nullptr, 0, dt, A, lda, B, ldb, s);
}

size_t factor_batch_table_bytes(int count) { return (size_t)count * sizeof(FacProb); }

size_t fac_static_bytes() { return sizeof(FacStatic); }

gptq2d_status upload_fac_static(Factors& f) {
  FacStatic s;
  s.f = fac_args(f);
  s.f.rev = 0;
  s.gpart = f.gpart;
  hipError_t e = hipMemcpy(f.d_fac, &s, sizeof(s), hipMemcpyHostToDevice);
  return e == hipSuccess ? GPTQ2D_OK : hip_fail(e, "handle upload");
}

gptq2d_status launch_factor_batched(int count, Factors* const* fs, gptq2d_dtype dt,
                                    const void* const* A, const int64_t* lda, const void* const* B,
                                    const int64_t* ldb, void* table, hipStream_t s) {
  static_assert(sizeof(FacProb) % sizeof(uint64_t) == 0, "the table is uploaded in 8-byte words");
  std::vector<FacProb> h(count);
  for (int p = 0; p < count; ++p)
    h[p] = FacProb{(const FacStatic*)fs[p]->d_fac, A[p], B[p], lda[p], ldb[p], fs[p]->rev};
  gptq2d_status st = enqueue_upload(table, h.data(), h.size() * sizeof(FacProb), s);
  if (st != GPTQ2D_OK) return st;
  return factor_impl(*fs[0], (const FacProb*)table, count, dt, nullptr, 0, nullptr, 0, s);
}

gptq2d_status launch_export(const Factors& f, double* L, int64_t ldl, double* U, int64_t ldu,
                            double* lamL, double* lamU, hipStream_t s) {
  const int bs = 256;
  if (L) {
    const int64_t tot = (int64_t)f.m * f.m;
    hipLaunchKernelGGL(k_export_tri, dim3((unsigned)((tot + bs - 1) / bs)), dim3(bs), 0, s, f.L,
                       f.mp, f.m, L, ldl, 1);
  }
  if (U) {
    const int64_t tot = (int64_t)f.n * f.n;
    hipLaunchKernelGGL(k_export_tri, dim3((unsigned)((tot + bs - 1) / bs)), dim3(bs), 0, s, f.U,
                       f.np, f.n, U, ldu, 0);
  }
  if (lamL) hipLaunchKernelGGL(k_export_lam, dim3((f.m + bs - 1) / bs), dim3(bs), 0, s, f.dL, f.m, lamL);
  if (lamU) hipLaunchKernelGGL(k_export_lam, dim3((f.n + bs - 1) / bs), dim3(bs), 0, s, f.dU, f.n, lamU);
  return check_launch("factor export");
}

gptq2d_status launch_import(Factors& f, const double* L, int64_t ldl, const double* U,
                            int64_t ldu, const double* lamL, const double* lamU, hipStream_t s) {
  const int bs = 256;
  int64_t tot = (int64_t)f.mp * f.mp;
  hipLaunchKernelGGL(k_import_tri, dim3((unsigned)((tot + bs - 1) / bs)), dim3(bs), 0, s, L, ldl,
                     f.m, f.mp, f.L, 1);
  tot = (int64_t)f.np * f.np;
  hipLaunchKernelGGL(k_import_tri, dim3((unsigned)((tot + bs - 1) / bs)), dim3(bs), 0, s, U, ldu,
                     f.n, f.np, f.U, 0);
  hipLaunchKernelGGL(k_import_lam, dim3((f.mp + bs - 1) / bs), dim3(bs), 0, s, lamL, f.m, f.mp, f.dL);
  hipLaunchKernelGGL(k_import_lam, dim3((f.np + bs - 1) / bs), dim3(bs), 0, s, lamU, f.n, f.np, f.dU);
  hipLaunchKernelGGL(k_zero_int, dim3(1), dim3(64), 0, s, f.flags, 1);
  return check_launch("factor import");
}

}  // namespace g2d
