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

// Lower-triangle enumeration of tile pairs: b -> (i, j) with i >= j.
__device__ __forceinline__ void tri_index(int b, int& i, int& j) {
  int r = (int)((sqrt(8.0 * (double)b + 1.0) - 1.0) * 0.5);
  while (r * (r + 1) / 2 > b) --r;
  while ((r + 1) * (r + 2) / 2 <= b) ++r;
  i = r;
  j = b - r * (r + 1) / 2;
}

// Gram operands with the index reversal folded in. The contraction index k
// runs over the rows of A (left Gram) or the columns of B (right Gram); the
// 64-wide index i is the reversed Gram index.
template <typename T>
struct OpGramLeft {  // element (i, k) = A[k][d-1-(i0+i)]
  const T* p;
  int64_t ld;
  int d, i0;
  __device__ __forceinline__ void fetch(int k0, double v[4]) const {
    const int t = threadIdx.x, k = k0 + (t >> 4), iq = (t & 15) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int idx = i0 + iq + e;
      v[e] = (idx < d && k < d) ? (double)p[(int64_t)k * ld + (d - 1 - idx)] : 0.0;
    }
  }
  __device__ __forceinline__ static void put(double (*s)[SA], const double v[4]) { OpKR::put(s, v); }
};

template <typename T>
struct OpGramRight {  // element (i, k) = B[d-1-(i0+i)][k]
  const T* p;
  int64_t ld;
  int d, i0;
  __device__ __forceinline__ void fetch(int k0, double v[4]) const {
    const int t = threadIdx.x, idx = i0 + (t >> 2), kq = k0 + (t & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = kq + e;
      v[e] = (idx < d && k < d) ? (double)p[(int64_t)(d - 1 - idx) * ld + k] : 0.0;
    }
  }
  __device__ __forceinline__ static void put(double (*s)[SA], const double v[4]) { OpRK::put(s, v); }
};

// Reversed Gram, lower tiles only, with an identity block on the padding.
template <typename T, int SIDE>
__global__ __launch_bounds__(NT) void k_gram(const T* S, int64_t ld, int d, int dp, double* gr) {
  __shared__ GemmSmem sm;
  int bp, bq;
  tri_index(blockIdx.x, bp, bq);
  Acc acc;
  acc.zero();
  if (SIDE == 0)
    gemm_acc(acc, OpGramLeft<T>{S, ld, d, bp * TB}, OpGramLeft<T>{S, ld, d, bq * TB}, dp, sm);
  else
    gemm_acc(acc, OpGramRight<T>{S, ld, d, bp * TB}, OpGramRight<T>{S, ld, d, bq * TB}, dp, sm);
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = bp * TB + acc_row(u, r), q = bq * TB + acc_col(v);
        double val = acc.t[2 * u + v][r];
        if (p >= d || q >= d) val = (p == q) ? 1.0 : 0.0;
        gr[(int64_t)p * dp + q] = val;
      }
}

// Cholesky of one 64 x 64 diagonal block (already updated by all previous
// panels) and the inverse of the resulting lower factor. Thread (c, g) with
// c = t & 63, g = t >> 6 keeps rows g, g+4, .., g+60 of column c in registers;
// each pivot step broadcasts one column through LDS (double-buffered, so two
// barriers per step). A pivot that is not positive and finite raises
// FLAG_SINGULAR and is replaced by 1 so that the remaining work stays finite.
__global__ __launch_bounds__(NT) void k_potrf_diag(double* gr, int dp, int kb, double* dinv,
                                                   int* flags) {
  __shared__ double S[TB][TB + 1];
  __shared__ double col[2][TB];
  const int t = threadIdx.x, c = t & 63, g = t >> 6;
  double* blk = gr + (int64_t)kb * TB * dp + (int64_t)kb * TB;
  double a[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) a[u] = blk[(int64_t)(g + 4 * u) * dp + c];
  for (int j = 0; j < TB; ++j) {
    double* cj = col[j & 1];
    if (c == j) {
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (g + 4 * u == j) {
          double piv = a[u];
          if (!(piv > 0.0) || !isfinite(piv)) {
            raise_flag(flags, FLAG_SINGULAR);
            piv = 1.0;
          }
          a[u] = sqrt(piv);
          cj[j] = a[u];
        }
      }
    }
    __syncthreads();
    if (c == j) {
      const double inv = 1.0 / cj[j];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int i = g + 4 * u;
        if (i > j) {
          a[u] *= inv;
          cj[i] = a[u];
        }
      }
    }
    __syncthreads();
    if (c > j) {
      const double cc = cj[c];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int i = g + 4 * u;
        if (i >= c) a[u] -= cj[i] * cc;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 16; ++u) S[g + 4 * u][c] = a[u];
  __syncthreads();
  // v = S^{-1}, right-looking by pivot rows; thread (c, g) keeps rows g+4u of
  // column c of the inverse (the pivot row is broadcast through a buffer that
  // alternates with k, so one barrier per row suffices).
  double v[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) v[u] = (g + 4 * u == c) ? 1.0 : 0.0;
  for (int k = 0; k < TB; ++k) {
    double* rk = col[k & 1];
    if ((k & 3) == g) {
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (4 * u + g == k) {
          v[u] = v[u] / S[k][k];
          rk[c] = v[u];
        }
    }
    __syncthreads();
    const double x = rk[c];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = g + 4 * u;
      if (i > k) v[u] -= S[i][k] * x;
    }
  }
  double* dv = dinv + (int64_t)kb * TB * TB;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int i = g + 4 * u;
    blk[(int64_t)i * dp + c] = (c <= i) ? a[u] : 0.0;
    dv[i * TB + c] = (c <= i) ? v[u] : 0.0;
  }
}

// Panel solve: Lc[ib][kb] = Q[ib][kb] * inv(Lc[kb][kb])^T for ib > kb.
__global__ __launch_bounds__(NT) void k_trsm(double* gr, int dp, int kb, const double* dinv) {
  __shared__ GemmSmem sm;
  const int ib = kb + 1 + blockIdx.x;
  double* blk = gr + (int64_t)ib * TB * dp + (int64_t)kb * TB;
  Acc acc;
  acc.zero();
  gemm_acc(acc, OpRK{blk, dp}, OpRK{dinv + (int64_t)kb * TB * TB, TB}, TB, sm);
  acc_store(acc, blk, dp, 1.0);
}

// Trailing update of the lower tiles: Q[bi][bj] -= Lc[bi][kb] Lc[bj][kb]^T.
__global__ __launch_bounds__(NT) void k_syrk(double* gr, int dp, int kb) {
  __shared__ GemmSmem sm;
  int bi, bj;
  tri_index(blockIdx.x, bi, bj);
  bi += kb + 1;
  bj += kb + 1;
  Acc acc;
  acc.zero();
  gemm_acc(acc, OpRK{gr + (int64_t)bi * TB * dp + (int64_t)kb * TB, dp},
           OpRK{gr + (int64_t)bj * TB * dp + (int64_t)kb * TB, dp}, TB, sm);
  double* out = gr + (int64_t)bi * TB * dp + (int64_t)bj * TB;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        double* p = out + (int64_t)acc_row(u, r) * dp + acc_col(v);
        *p = *p - acc.t[2 * u + v][r];
      }
}

// Blocked triangular inverse Li = Lc^{-1}, row block kb: Li[kb][kb] = dinv[kb];
// Li[kb][jb] = -dinv[kb] * S[kb][jb] (jb < kb), where S[kb][jb] =
// sum_{j <= k < kb} Lc[kb][k] Li[k][jb] has been accumulated in place.
__global__ __launch_bounds__(NT) void k_trtri_row(double* li, int dp, int kb, const double* dinv) {
  __shared__ GemmSmem sm;
  const int jb = blockIdx.x;
  double* out = li + (int64_t)kb * TB * dp + (int64_t)jb * TB;
  const double* dk = dinv + (int64_t)kb * TB * TB;
  if (jb == kb) {
    for (int e = threadIdx.x; e < TB * TB; e += NT) out[(int64_t)(e >> 6) * dp + (e & 63)] = dk[e];
    return;
  }
  Acc acc;
  acc.zero();
  gemm_acc(acc, OpRK{dk, TB}, OpKR{out, dp}, TB, sm);
  acc_store(acc, out, dp, -1.0);
}

// S[ib][jb] += Lc[ib][kb] Li[kb][jb] for ib > kb, jb <= kb (the first
// contribution, kb == jb, overwrites).
__global__ __launch_bounds__(NT) void k_trtri_upd(double* li, const double* gr, int dp, int kb) {
  __shared__ GemmSmem sm;
  const int w = kb + 1;
  const int ib = kb + 1 + blockIdx.x / w, jb = blockIdx.x % w;
  Acc acc;
  acc.zero();
  gemm_acc(acc, OpRK{gr + (int64_t)ib * TB * dp + (int64_t)kb * TB, dp},
           OpKR{li + (int64_t)kb * TB * dp + (int64_t)jb * TB, dp}, TB, sm);
  double* out = li + (int64_t)ib * TB * dp + (int64_t)jb * TB;
  if (jb != kb) acc_add_from(acc, out, dp);
  acc_store(acc, out, dp, 1.0);
}

// Normalisation into the feedback factor (side 0: L, lower; side 1: U, upper)
// and the diagonal 1/Lambda. One workgroup per output tile of the kept
// triangle; the padding becomes an identity block.
__global__ __launch_bounds__(NT) void k_finalize(const double* lc, const double* li, int d, int dp,
                                                 double* out, double* dout, int side) {
  __shared__ double S[TB][TB + 1];
  __shared__ double sc[TB];
  int bi, bj;
  tri_index(blockIdx.x, bi, bj);  // bi >= bj
  const int rs = d - TB - bj * TB, cs = d - TB - bi * TB;
  const int t = threadIdx.x;
  for (int e = t; e < TB * TB; e += NT) {
    const int x = e >> 6, y = e & 63, r = rs + x, c = cs + y;
    S[x][y] = (r >= 0 && r < d && c >= 0 && c < d) ? li[(int64_t)r * dp + c] : 0.0;
  }
  if (t < TB) {
    const int r = rs + t;
    sc[t] = (r >= 0 && r < d) ? lc[(int64_t)r * dp + r] : 1.0;
  }
  __syncthreads();
  // side 0: tile (bi, bj), element (bi*64+a, bj*64+b) = S[63-b][63-a] * sc[63-b]
  // side 1: tile (bj, bi), element (bj*64+a, bi*64+b) = S[63-a][63-b] * sc[63-a]
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
    out[(int64_t)i * dp + j] = val;
  }
  if (bi == bj && t < TB) {
    const int i = bi * TB + t;
    dout[i] = (i < d) ? sc[63 - t] * sc[63 - t] : 1.0;
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

template <typename T, int SIDE>
static gptq2d_status factor_side(Factors& f, const T* S, int64_t ld, hipStream_t s) {
  const int d = SIDE == 0 ? f.m : f.n;
  const int dp = SIDE == 0 ? f.mp : f.np;
  const int nb = dp / TB;
  double* gr = f.gram[SIDE];
  double* li = f.inv[SIDE];
  double* dinv = f.dinv[SIDE];
  hipLaunchKernelGGL((k_gram<T, SIDE>), dim3(nb * (nb + 1) / 2), dim3(NT), 0, s, S, ld, d, dp, gr);
  for (int kb = 0; kb < nb; ++kb) {
    hipLaunchKernelGGL(k_potrf_diag, dim3(1), dim3(NT), 0, s, gr, dp, kb, dinv, f.flags);
    const int rest = nb - kb - 1;
    if (rest > 0) {
      hipLaunchKernelGGL(k_trsm, dim3(rest), dim3(NT), 0, s, gr, dp, kb, dinv);
      hipLaunchKernelGGL(k_syrk, dim3(rest * (rest + 1) / 2), dim3(NT), 0, s, gr, dp, kb);
    }
  }
  for (int kb = 0; kb < nb; ++kb) {
    hipLaunchKernelGGL(k_trtri_row, dim3(kb + 1), dim3(NT), 0, s, li, dp, kb, dinv);
    const int rest = nb - kb - 1;
    if (rest > 0)
      hipLaunchKernelGGL(k_trtri_upd, dim3(rest * (kb + 1)), dim3(NT), 0, s, li, gr, dp, kb);
  }
  hipLaunchKernelGGL(k_finalize, dim3(nb * (nb + 1) / 2), dim3(NT), 0, s, gr, li, d, dp,
                     SIDE == 0 ? f.L : f.U, SIDE == 0 ? f.dL : f.dU, SIDE);
  return check_launch("factorisation launch");
}

gptq2d_status launch_factor(Factors& f, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_int, dim3(1), dim3(64), 0, s, f.flags, 1);
  gptq2d_status st;
  if (dt == GPTQ2D_F32) {
    st = factor_side<float, 0>(f, (const float*)A, lda, s);
    if (st == GPTQ2D_OK) st = factor_side<float, 1>(f, (const float*)B, ldb, s);
  } else {
    st = factor_side<double, 0>(f, (const double*)A, lda, s);
    if (st == GPTQ2D_OK) st = factor_side<double, 1>(f, (const double*)B, ldb, s);
  }
  return st;
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
