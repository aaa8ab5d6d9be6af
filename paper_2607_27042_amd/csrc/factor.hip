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
};

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
__device__ __forceinline__ void gram_load(const T* S, int64_t ld, int d, int i0, int k0, double r[16]) {
  const int t = threadIdx.x;
  T v[16];
  bool ok[16];
  // unconditional loads from clamped addresses (no per-load branch), then
  // zero what lies outside the matrix
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s, hi = e >> 6, lo = e & 63;
    int64_t off;
    if (SIDE == 0) {  // (k = hi, i = lo): A[k0+k][d-1-(i0+i)], coalesced along i
      const int k = k0 + hi, idx = i0 + lo;
      ok[s] = k < d && idx < d;
      off = (int64_t)k * ld + (d - 1 - idx);
    } else {          // (i = hi, k = lo): B[d-1-(i0+i)][k0+k], coalesced along k
      const int idx = i0 + hi, k = k0 + lo;
      ok[s] = k < d && idx < d;
      off = (int64_t)(d - 1 - idx) * ld + k;
    }
    v[s] = S[ok[s] ? off : 0];
  }
#pragma unroll
  for (int s = 0; s < 16; ++s) r[s] = ok[s] ? (double)v[s] : 0.0;
}

template <typename T, int SIDE>
__device__ void gram_tile(const Side& sd, const T* S, int64_t ld, int bp, int bq, Stage64& st) {
  Acc acc;
  acc.zero();
  double ra[16], rb[16];
  gram_load<T, SIDE>(S, ld, sd.d, bp * TB, 0, ra);
  gram_load<T, SIDE>(S, ld, sd.d, bq * TB, 0, rb);
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
      gram_load<T, SIDE>(S, ld, sd.d, bp * TB, (kb + 1) * TB, ra);
      gram_load<T, SIDE>(S, ld, sd.d, bq * TB, (kb + 1) * TB, rb);
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

template <typename T>
__global__ __launch_bounds__(NT) void k_gram(FacArgs f, const T* A, int64_t lda, const T* B,
                                             int64_t ldb) {
  __shared__ Stage64 st;
  const int t0 = f.s[0].nb * (f.s[0].nb + 1) / 2;
  int bp, bq;
  if ((int)blockIdx.x < t0) {
    tri_index(blockIdx.x, bp, bq);
    gram_tile<T, 0>(f.s[0], A, lda, bp, bq, st);
  } else {
    tri_index(blockIdx.x - t0, bp, bq);
    gram_tile<T, 1>(f.s[1], B, ldb, bp, bq, st);
  }
}

// ---------------------------------------------------------------------------
// Cholesky of one 64 x 64 diagonal block (already updated by all earlier
// panels) and the inverse of its lower factor; one workgroup per side.
// Thread (c, g), c = t & 63, g = t >> 6, keeps rows g + 4u of column c in
// registers. The pivot loops are unrolled so every register index is a
// constant; each pivot column / row is broadcast through a buffer that
// alternates between steps. A pivot that is not positive and finite raises
// FLAG_SINGULAR and is replaced by 1 so the remaining work stays finite.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(NT) void k_diag(FacArgs f, int kb) {
  const Side& sd = f.s[blockIdx.x];
  if (kb >= sd.nb) return;
  __shared__ double S[TB][TB + 1];
  __shared__ double col[2][TB];
  __shared__ double rd[TB];
  const int t = threadIdx.x, c = t & 63, g = t >> 6;
  double* blk = sd.gr + (int64_t)kb * TB * sd.dp + (int64_t)kb * TB;
  // a[u] is entry (g + 4u, c); the upper triangle starts at zero. Updates are
  // applied to every row of a thread without masking: entries above the
  // diagonal collect finite junk that no valid entry ever reads, and they are
  // written out as zero.
  double a[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const double x = blk[(int64_t)(g + 4 * u) * sd.dp + c];
    a[u] = (g + 4 * u >= c) ? x : 0.0;
  }
#pragma unroll 1
  for (int j = 0; j < TB; ++j) {
    double* cj = col[j & 1];
    if (c == j) {  // publish column j before its scaling; cj[j] is the pivot
#pragma unroll
      for (int u = 0; u < 16; ++u) cj[g + 4 * u] = a[u];
    }
    __syncthreads();
    double piv = cj[j];
    if (!(piv > 0.0) || !isfinite(piv)) {
      if (t == 0) raise_flag(f.flags, FLAG_SINGULAR);
      piv = 1.0;
    }
    if (c == j) {  // L[i][j] = a_ij / sqrt(piv)
      const double rsq = 1.0 / sqrt(piv);
#pragma unroll
      for (int u = 0; u < 16; ++u) a[u] *= rsq;
    } else if (c > j) {  // a_ic -= L[i][j] L[c][j] = a_ij a_cj / piv
      const double cc = cj[c] / piv;
#pragma unroll
      for (int u = 0; u < 16; ++u) a[u] = fma(-cj[g + 4 * u], cc, a[u]);
    }
  }
  // Lc into LDS: strictly lower part in S, reciprocal of the diagonal in rd
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int i = g + 4 * u;
    S[i][c] = (c < i) ? a[u] : 0.0;
    if (c == i) rd[i] = 1.0 / a[u];
    blk[(int64_t)i * sd.dp + c] = (c <= i) ? a[u] : 0.0;
  }
  __syncthreads();
  // V = Lc^{-1} by forward substitution on the identity, one pivot row per
  // step; v[u] holds row g + 4(u + U) of column c (window shifting with U);
  // rows past the block hold finite junk and are never stored.
  double* dv = sd.dinv + (int64_t)kb * TB * TB;
  double v[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) v[u] = (g + 4 * u == c) ? 1.0 : 0.0;
#pragma unroll 1
  for (int U = 0; U < 16; ++U) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int k = 4 * U + kk;
      double* rk = col[kk & 1];
      if (g == kk) {
        v[0] *= rd[k];
        rk[c] = v[0];
      }
      __syncthreads();
      const double x = rk[c];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = fma(-S[(g + 4 * (u + U)) & 63][k], x, v[u]);
    }
    const int i = g + 4 * U;
    dv[i * TB + c] = (c <= i) ? v[0] : 0.0;
#pragma unroll
    for (int u = 0; u < 15; ++u) v[u] = v[u + 1];
  }
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

__global__ __launch_bounds__(NT) void k_panel(FacArgs f, int kb) {
  __shared__ Stage64 st;
  int b = blockIdx.x;
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
// Update step kb, both sides in one grid:
//   Q[bi][bj] -= Lc[bi][kb] Lc[bj][kb]^T          (kb < bj <= bi)
//   S[ib][jb] += Lc[ib][kb] Li[kb][jb]            (ib > kb, jb <= kb; kb == jb overwrites)
// ---------------------------------------------------------------------------

__device__ __forceinline__ int update_count(const Side& sd, int kb) {
  if (kb >= sd.nb) return 0;
  const int rest = sd.nb - kb - 1;
  return rest * (rest + 1) / 2 + rest * (kb + 1);
}

__global__ __launch_bounds__(NT) void k_update(FacArgs f, int kb) {
  __shared__ Stage64 st;
  int b = blockIdx.x;
  const int n0 = update_count(f.s[0], kb);
  const Side& sd = (b < n0) ? f.s[0] : f.s[1];
  if (b >= n0) b -= n0;
  const int rest = sd.nb - kb - 1;
  const int nsyrk = rest * (rest + 1) / 2;
  Acc acc;
  acc.zero();
  if (b < nsyrk) {
    int bi, bj;
    tri_index(b, bi, bj);
    bi += kb + 1;
    bj += kb + 1;
    gemm64<1>(acc, sd.gr + (int64_t)bi * TB * sd.dp + (int64_t)kb * TB, sd.dp,
              sd.gr + (int64_t)bj * TB * sd.dp + (int64_t)kb * TB, sd.dp, st);
    double* out = sd.gr + (int64_t)bi * TB * sd.dp + (int64_t)bj * TB;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          double* q = out + (int64_t)acc_row(u, r) * sd.dp + acc_col(v);
          *q = *q - acc.t[2 * u + v][r];
        }
  } else {
    b -= nsyrk;
    const int w = kb + 1, ib = kb + 1 + b / w, jb = b % w;
    double* out = sd.li + (int64_t)ib * TB * sd.dp + (int64_t)jb * TB;
    if (jb != kb) acc_add_from(acc, out, sd.dp);
    gemm64<0>(acc, sd.gr + (int64_t)ib * TB * sd.dp + (int64_t)kb * TB, sd.dp,
              sd.li + (int64_t)kb * TB * sd.dp + (int64_t)jb * TB, sd.dp, st);
    acc_store(acc, out, sd.dp, 1.0);
  }
}

// ---------------------------------------------------------------------------
// Normalisation into the feedback factor and 1/Lambda (both sides):
//   side 0: L[i][j] = Li[d-1-j][d-1-i] Lc[d-1-j][d-1-j]  (i > j), lower tiles
//   side 1: U[i][j] = Li[d-1-i][d-1-j] Lc[d-1-i][d-1-i]  (j > i), upper tiles
//   1/Lambda[i] = Lc[d-1-i][d-1-i]^2; the padding becomes an identity block.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(NT) void k_finalize(FacArgs f) {
  __shared__ double S[TB][TB + 1];
  __shared__ double sc[TB];
  const int t0 = f.s[0].nb * (f.s[0].nb + 1) / 2;
  const int side = (int)blockIdx.x < t0 ? 0 : 1;
  const Side& sd = f.s[side];
  int bi, bj;
  tri_index(side == 0 ? blockIdx.x : blockIdx.x - t0, bi, bj);  // bi >= bj
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
    sd.out[(int64_t)i * dp + j] = val;
  }
  if (bi == bj && t < TB) {
    const int i = bi * TB + t;
    sd.dout[i] = (i < d) ? sc[63 - t] * sc[63 - t] : 1.0;
  }
}

__global__ void k_zero_int(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// factor export: dense triangle out of the padded storage, lam = 1 / dl.
__global__ void k_export_tri(const double* src, int dp, int d, double* dst, int64_t ld, int lower) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)d * d) return;
  const int i = (int)(e / d), j = (int)(e % d);
  const bool keep = lower ? (j <= i) : (j >= i);
  dst[(int64_t)i * ld + j] = keep ? (i == j ? 1.0 : src[(int64_t)i * dp + j]) : 0.0;
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
  dst[e] = v;
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
  return a;
}

static int h_panel_count(int nb, int kb) { return kb < nb ? nb : 0; }
static int h_update_count(int nb, int kb) {
  if (kb >= nb) return 0;
  const int rest = nb - kb - 1;
  return rest * (rest + 1) / 2 + rest * (kb + 1);
}

gptq2d_status launch_factor(Factors& f, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, hipStream_t s) {
  FacArgs a = fac_args(f);
  const int nb0 = a.s[0].nb, nb1 = a.s[1].nb, nbmax = nb0 > nb1 ? nb0 : nb1;
  const int tri = nb0 * (nb0 + 1) / 2 + nb1 * (nb1 + 1) / 2;
  hipLaunchKernelGGL(k_zero_int, dim3(1), dim3(64), 0, s, f.flags, 1);
  if (dt == GPTQ2D_F32)
    hipLaunchKernelGGL(k_gram<float>, dim3(tri), dim3(NT), 0, s, a, (const float*)A, lda,
                       (const float*)B, ldb);
  else
    hipLaunchKernelGGL(k_gram<double>, dim3(tri), dim3(NT), 0, s, a, (const double*)A, lda,
                       (const double*)B, ldb);
  for (int kb = 0; kb < nbmax; ++kb) {
    hipLaunchKernelGGL(k_diag, dim3(2), dim3(NT), 0, s, a, kb);
    const int np_ = h_panel_count(nb0, kb) + h_panel_count(nb1, kb);
    if (np_ > 0) hipLaunchKernelGGL(k_panel, dim3(np_), dim3(NT), 0, s, a, kb);
    const int nu = h_update_count(nb0, kb) + h_update_count(nb1, kb);
    if (nu > 0) hipLaunchKernelGGL(k_update, dim3(nu), dim3(NT), 0, s, a, kb);
  }
  hipLaunchKernelGGL(k_finalize, dim3(tri), dim3(NT), 0, s, a);
  return check_launch("factorisation launch");
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
