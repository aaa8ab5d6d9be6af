/*
 * CPU oracle for two-sided adaptive rounding (GPTQ-2D, arXiv 2607.27042).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline leg
 * of the benchmark do. It shares no code, header, table or helper with the GPU
 * path.
 *
 * Everything here is plain, slow, double precision, written for a reader who
 * checks it against the paper by eye:
 *   - Gram matrices by their definition (Sec. 3.2, Eq. GH),
 *   - feedback factors by the paper's literal route: invert the Gram, then take
 *     the unit-lower LDL factor of the inverse (Sec. 3.1, and the first two
 *     steps of every algorithm),
 *   - Algorithm 1 (one-dimensional adaptive rounding), applied either to an
 *     explicit Kronecker Gram H (x) G over the column-major vectorisation
 *     (Sec. 3.2, Eq. kron-objective) -- quartic -- or with the vectorised
 *     feedback F = U^T (x) L generated column by column (Eq.
 *     vectorized-feedback),
 *   - Algorithm 5 (nested column-major form, Appendix A) -- cubic,
 *   - Algorithm 3 (GPTQ-2D, Sec. 4.2) and Algorithm 6 (implicit-Y form,
 *     Appendix B) as cross-checks,
 *   - the objective ||A (Z - X) B||_F^2 by its definition (Eq. objective).
 *
 * Readings taken where the paper is silent:
 *   - the nearest-integer operator breaks ties to even (C nearbyint in the
 *     default FE_TONEAREST mode); the paper only asks for a deterministic rule
 *     (Theorem 1);
 *   - the "corrected value" reported for an entry is y at the moment it is
 *     rounded;
 *   - Z is stored as int32; a value outside the int32 range is an error.
 *
 * Synchronised replay: every sweep accepts an optional hint matrix Zh and a
 * window tau. When the oracle's own rounding disagrees with the hint, the entry
 * is counted as a "window" entry if y lies within tau of the half-integer
 * between the two candidates, otherwise as a "hard" mismatch; in both cases the
 * hint is adopted so that the replay stays on the hinted trajectory.
 *
 * Storage: all matrices row-major, X is m x n, A is m x m, B is n x n, L is
 * m x m unit lower, U is n x n unit upper.
 */
#include <fenv.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_SINGULAR (-2)
#define ORC_ERR_RANGE (-7)
#define ORC_ERR_NOMEM (-4)

/* ------------------------------------------------------------------------ */
/* Gram matrices (Sec. 3.2, Eq. GH)                                          */
/* ------------------------------------------------------------------------ */

/* G = A^T A, A is m x m. */
void orc_gram_left(int m, const double* A, double* G) {
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < m; ++i) {
    for (int j = 0; j < m; ++j) {
      long double s = 0.0L;
      for (int k = 0; k < m; ++k) s += (long double)A[(size_t)k * m + i] * A[(size_t)k * m + j];
      G[(size_t)i * m + j] = (double)s;
    }
  }
}

/* H = B B^T, B is n x n. */
void orc_gram_right(int n, const double* B, double* H) {
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < n; ++i) {
    for (int j = 0; j < n; ++j) {
      long double s = 0.0L;
      for (int k = 0; k < n; ++k) s += (long double)B[(size_t)i * n + k] * B[(size_t)j * n + k];
      H[(size_t)i * n + j] = (double)s;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* Inverse and LDL (Sec. 3.1: the feedback is the unit-lower LDL factor of   */
/* the inverse Gram)                                                         */
/* ------------------------------------------------------------------------ */

/* Gauss-Jordan elimination with partial pivoting on [M | I]. */
int orc_inverse(int d, const double* M, double* Minv) {
  size_t w = 2 * (size_t)d;
  double* T = (double*)malloc(sizeof(double) * (size_t)d * w);
  if (!T) return ORC_ERR_NOMEM;
  for (int i = 0; i < d; ++i) {
    for (int j = 0; j < d; ++j) {
      T[i * w + j] = M[(size_t)i * d + j];
      T[i * w + d + j] = (i == j) ? 1.0 : 0.0;
    }
  }
  for (int c = 0; c < d; ++c) {
    int p = c;
    double best = fabs(T[(size_t)c * w + c]);
    for (int r = c + 1; r < d; ++r) {
      double v = fabs(T[(size_t)r * w + c]);
      if (v > best) { best = v; p = r; }
    }
    if (!(best > 0.0) || !isfinite(best)) { free(T); return ORC_ERR_SINGULAR; }
    if (p != c) {
      for (size_t j = 0; j < w; ++j) {
        double t = T[(size_t)c * w + j];
        T[(size_t)c * w + j] = T[(size_t)p * w + j];
        T[(size_t)p * w + j] = t;
      }
    }
    double piv = T[(size_t)c * w + c];
    for (size_t j = 0; j < w; ++j) T[(size_t)c * w + j] /= piv;
#pragma omp parallel for schedule(static)
    for (int r = 0; r < d; ++r) {
      if (r == c) continue;
      double f = T[(size_t)r * w + c];
      if (f == 0.0) continue;
      /* columns left of c are already reduced to unit vectors, and row c is
         zero there, so the elimination only has to touch columns >= c */
      for (size_t j = (size_t)c; j < w; ++j) T[(size_t)r * w + j] -= f * T[(size_t)c * w + j];
    }
  }
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < d; ++j) Minv[(size_t)i * d + j] = T[(size_t)i * w + d + j];
  free(T);
  return ORC_OK;
}

/* S = F diag(D) F^T with F unit lower triangular (textbook LDL^T, column by
 * column). Only the lower triangle of S is read. */
int orc_ldl(int d, const double* S, double* F, double* D) {
  memset(F, 0, sizeof(double) * (size_t)d * d);
  for (int j = 0; j < d; ++j) {
    double dj = S[(size_t)j * d + j];
    for (int k = 0; k < j; ++k) dj -= F[(size_t)j * d + k] * F[(size_t)j * d + k] * D[k];
    if (!(dj > 0.0) || !isfinite(dj)) return ORC_ERR_SINGULAR;
    D[j] = dj;
    F[(size_t)j * d + j] = 1.0;
#pragma omp parallel for schedule(static)
    for (int i = j + 1; i < d; ++i) {
      double s = S[(size_t)i * d + j];
      for (int k = 0; k < j; ++k) s -= F[(size_t)i * d + k] * F[(size_t)j * d + k] * D[k];
      F[(size_t)i * d + j] = s / dj;
    }
  }
  return ORC_OK;
}

/* Feedback factor of one quadratic metric (Sec. 3.1): with Gram matrix Q,
 * Q^{-1} = F Lambda F^T, F unit lower. */
int orc_feedback(int d, const double* Q, double* F, double* lam) {
  double* Qi = (double*)malloc(sizeof(double) * (size_t)d * d);
  if (!Qi) return ORC_ERR_NOMEM;
  int st = orc_inverse(d, Q, Qi);
  if (st == ORC_OK) st = orc_ldl(d, Qi, F, lam);
  free(Qi);
  return st;
}

/* Per-axis factors of the two-sided problem (Sec. 4.1):
 *   L unit lower with (A^T A)^{-1} = L diag(lamL) L^T,
 *   U unit upper with (B B^T)^{-1} = U^T diag(lamU) U,
 * i.e. U is the transpose of the LDL factor of the inverse right Gram. */
int orc_factors(int m, int n, const double* A, const double* B, double* L, double* lamL,
                double* U, double* lamU) {
  double* G = (double*)malloc(sizeof(double) * (size_t)m * m);
  double* H = (double*)malloc(sizeof(double) * (size_t)n * n);
  double* Ft = (double*)malloc(sizeof(double) * (size_t)n * n);
  int st = ORC_ERR_NOMEM;
  if (G && H && Ft) {
    orc_gram_left(m, A, G);
    orc_gram_right(n, B, H);
    st = orc_feedback(m, G, L, lamL);
    if (st == ORC_OK) st = orc_feedback(n, H, Ft, lamU);
    if (st == ORC_OK)
      for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) U[(size_t)i * n + j] = Ft[(size_t)j * n + i];
  }
  free(G);
  free(H);
  free(Ft);
  return st;
}

/* ------------------------------------------------------------------------ */
/* The rounding decision shared by every sweep below                         */
/* ------------------------------------------------------------------------ */

typedef struct {
  const int32_t* hint; /* nullable: synchronised-replay hint, indexed like Z */
  double tau;          /* half-width of the tie window around a half-integer */
  int64_t* counts;     /* [0] window entries, [1] hard mismatches, [2] range errors */
  int64_t* hard_idx;   /* first hard mismatches (flat index into Z) */
  int hard_cap;
} orc_replay;

/* Nearest integer of y with ties to even; in replay mode the hint wins. */
static double orc_decide(double y, size_t zidx, const orc_replay* rp) {
  double z = nearbyint(y);
  if (rp && rp->hint) {
    double h = (double)rp->hint[zidx];
    if (z != h) {
      if (fabs(z - h) == 1.0 && fabs(y - 0.5 * (z + h)) <= rp->tau) {
        rp->counts[0] += 1;
      } else {
        if (rp->counts[1] < rp->hard_cap) rp->hard_idx[rp->counts[1]] = (int64_t)zidx;
        rp->counts[1] += 1;
      }
      z = h;
    }
  }
  return z;
}

static int32_t orc_to_int(double z, const orc_replay* rp, int* bad) {
  if (!(z >= -2147483648.0 && z <= 2147483647.0)) {
    *bad = 1;
    if (rp && rp->counts) rp->counts[2] += 1;
    return 0;
  }
  return (int32_t)z;
}

static void orc_replay_init(orc_replay* rp, const int32_t* hint, double tau, int64_t* counts,
                            int64_t* hard_idx, int hard_cap) {
  rp->hint = hint;
  rp->tau = tau;
  rp->counts = counts;
  rp->hard_idx = hard_idx;
  rp->hard_cap = hard_idx ? hard_cap : 0;
  if (counts) counts[0] = counts[1] = counts[2] = 0;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1: one-dimensional adaptive rounding                            */
/* ------------------------------------------------------------------------ */

/* x, z, ypre have length d; F is d x d unit lower triangular (row-major).
 * zmap (nullable) maps the sweep position k to the index used for the hint
 * and for z/ypre; identity when NULL. */
static int orc_sweep_1d(int64_t d, const double* x, const double* F, const int64_t* zmap,
                        const orc_replay* rp, int32_t* z, double* ypre) {
  double* y = (double*)malloc(sizeof(double) * (size_t)d);
  if (!y) return ORC_ERR_NOMEM;
  memcpy(y, x, sizeof(double) * (size_t)d);
  int bad = 0;
  for (int64_t k = 0; k < d; ++k) {
    size_t o = zmap ? (size_t)zmap[k] : (size_t)k;
    double yk = y[k];
    double zk = orc_decide(yk, o, rp);
    double e = zk - yk;
    z[o] = orc_to_int(zk, rp, &bad);
    ypre[o] = yk;
#pragma omp parallel for schedule(static) if (d - k > 4096)
    for (int64_t l = k; l < d; ++l) y[l] += F[(size_t)l * d + k] * e;
  }
  free(y);
  return bad ? ORC_ERR_RANGE : ORC_OK;
}

int orc_round_1d(int d, const double* x, const double* F, const int32_t* hint, double tau,
                 int32_t* z, double* ypre, int64_t* counts, int64_t* hard_idx, int hard_cap) {
  orc_replay rp;
  int64_t local[3];
  orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
  return orc_sweep_1d(d, x, F, NULL, &rp, z, ypre);
}

/* Quartic route: form the Kronecker Gram K = H (x) G of the column-major
 * vectorisation (Eq. kron-objective), take its feedback factor by the generic
 * 1-D construction, and run Algorithm 1 on vec(X). Nothing about the
 * per-axis factors is assumed. Memory (mn)^2 doubles twice: small sizes only. */
int orc_round_quartic(int m, int n, const double* X, const double* A, const double* B,
                      const int32_t* hint, double tau, int32_t* Z, double* Ypre,
                      int64_t* counts, int64_t* hard_idx, int hard_cap) {
  int64_t d = (int64_t)m * n;
  double* G = (double*)malloc(sizeof(double) * (size_t)m * m);
  double* H = (double*)malloc(sizeof(double) * (size_t)n * n);
  double* K = (double*)malloc(sizeof(double) * (size_t)(d * d));
  double* F = (double*)malloc(sizeof(double) * (size_t)(d * d));
  double* lam = (double*)malloc(sizeof(double) * (size_t)d);
  double* x = (double*)malloc(sizeof(double) * (size_t)d);
  int64_t* zmap = (int64_t*)malloc(sizeof(int64_t) * (size_t)d);
  int st = ORC_ERR_NOMEM;
  if (G && H && K && F && lam && x && zmap) {
    orc_gram_left(m, A, G);
    orc_gram_right(n, B, H);
    /* vec index k = j*m + i  <->  entry (i, j) */
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < d; ++r) {
      int64_t jr = r / m, ir = r % m;
      for (int64_t c = 0; c < d; ++c) {
        int64_t jc = c / m, ic = c % m;
        K[(size_t)(r * d + c)] = H[(size_t)jr * n + jc] * G[(size_t)ir * m + ic];
      }
    }
    st = orc_feedback((int)d, K, F, lam);
    if (st == ORC_OK) {
      for (int64_t k = 0; k < d; ++k) {
        int64_t j = k / m, i = k % m;
        x[k] = X[(size_t)i * n + j];
        zmap[k] = i * n + j;
      }
      orc_replay rp;
      int64_t local[3];
      orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
      st = orc_sweep_1d(d, x, F, zmap, &rp, Z, Ypre);
    }
  }
  free(G);
  free(H);
  free(K);
  free(F);
  free(lam);
  free(x);
  free(zmap);
  return st;
}

/* Algorithm 1 over vec(X) with the vectorised feedback F = U^T (x) L of
 * Eq. vectorized-feedback, generated entry by entry from the per-axis factors:
 * F[(j2 m + i2), (j m + i)] = U[j][j2] * L[i2][i]. Quartic work, O(mn) memory. */
int orc_round_kron(int m, int n, const double* X, const double* L, const double* U,
                   const int32_t* hint, double tau, int32_t* Z, double* Ypre, int64_t* counts,
                   int64_t* hard_idx, int hard_cap) {
  int64_t d = (int64_t)m * n;
  double* y = (double*)malloc(sizeof(double) * (size_t)d);
  if (!y) return ORC_ERR_NOMEM;
  for (int64_t k = 0; k < d; ++k) y[k] = X[(size_t)(k % m) * n + (size_t)(k / m)];
  orc_replay rp;
  int64_t local[3];
  orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
  int bad = 0;
  for (int64_t k = 0; k < d; ++k) {
    int j = (int)(k / m), i = (int)(k % m);
    size_t o = (size_t)i * n + j;
    double yk = y[k];
    double zk = orc_decide(yk, o, &rp);
    double e = zk - yk;
    Z[o] = orc_to_int(zk, &rp, &bad);
    Ypre[o] = yk;
    /* y_{k:d} += F_{k:d,k} e; F is zero above row k inside column j (L lower). */
#pragma omp parallel for schedule(static) if ((int64_t)(n - j) * (m - i) > 65536)
    for (int j2 = j; j2 < n; ++j2) {
      double u = U[(size_t)j * n + j2];
      if (u == 0.0) continue;
      int i2s = (j2 == j) ? i : 0;
      for (int i2 = i2s; i2 < m; ++i2) y[(size_t)j2 * m + i2] += u * L[(size_t)i2 * m + i] * e;
    }
  }
  free(y);
  return bad ? ORC_ERR_RANGE : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 5: nested column-major form (Appendix A) -- the cubic oracle    */
/* ------------------------------------------------------------------------ */

/* Algorithm 5 on the first ncols columns only (0 <= ncols <= n): the sweep is
 * column by column and an error at (i, j) reaches only columns >= j (Eq.
 * rank-one-update), so these columns of Z and Ypre are those of the whole
 * sweep; the later columns of Z and Ypre are left unwritten. This bounds the
 * CPU work of a large problem for timing. */
int orc_round_nested_cols(int m, int n, int ncols, const double* X, const double* L, const double* U,
                          const int32_t* hint, double tau, int32_t* Z, double* Ypre, int64_t* counts,
                          int64_t* hard_idx, int hard_cap) {
  if (ncols < 0 || ncols > n) return ORC_ERR_RANGE;
  double* Y = (double*)malloc(sizeof(double) * (size_t)m * n);
  double* y = (double*)malloc(sizeof(double) * (size_t)m);
  if (!Y || !y) { free(Y); free(y); return ORC_ERR_NOMEM; }
  memcpy(Y, X, sizeof(double) * (size_t)m * n);
  orc_replay rp;
  int64_t local[3];
  orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
  int bad = 0;
  for (int j = 0; j < ncols; ++j) {
    /* y <- Y[:, j]; one-dimensional sweep of the column under L */
    for (int i = 0; i < m; ++i) y[i] = Y[(size_t)i * n + j];
    for (int i = 0; i < m; ++i) {
      size_t o = (size_t)i * n + j;
      double yi = y[i];
      double zi = orc_decide(yi, o, &rp);
      double e = zi - yi;
      Z[o] = orc_to_int(zi, &rp, &bad);
      Ypre[o] = yi;
      for (int l = i; l < m; ++l) y[l] += L[(size_t)l * m + i] * e;
    }
    /* Y <- Y + (y - Y[:, j]) U[j, :]; U[j, q] = 0 for q < j, so start at j. */
#pragma omp parallel for schedule(static) if ((int64_t)m * (n - j) > 65536)
    for (int i = 0; i < m; ++i) {
      double* row = Y + (size_t)i * n;
      double dcol = y[i] - row[j];
      const double* urow = U + (size_t)j * n;
      for (int q = j; q < n; ++q) row[q] += dcol * urow[q];
    }
  }
  free(Y);
  free(y);
  return bad ? ORC_ERR_RANGE : ORC_OK;
}

int orc_round_nested(int m, int n, const double* X, const double* L, const double* U,
                     const int32_t* hint, double tau, int32_t* Z, double* Ypre, int64_t* counts,
                     int64_t* hard_idx, int hard_cap) {
  return orc_round_nested_cols(m, n, n, X, L, U, hint, tau, Z, Ypre, counts, hard_idx, hard_cap);
}

/* Nested form restricted to the leading block rows [0, m1) x columns [0, n1):
 * that block depends on nothing outside itself (Eq. rank-one-update: an error
 * at (i, j) reaches only rows >= i and columns >= j), so its trajectory is the
 * trajectory of the full problem there. Used to check large outputs on a
 * corner the CPU can afford. Arguments keep the full problem's leading
 * dimensions: X has row stride n, L row stride m, U row stride n; Z, Ypre and
 * the hint are m1 x n1 with row stride n1. */
int orc_round_nested_corner(int m, int n, int m1, int n1, const double* X, const double* L,
                            const double* U, const int32_t* hint, double tau, int32_t* Z,
                            double* Ypre, int64_t* counts, int64_t* hard_idx, int hard_cap) {
  double* Xc = (double*)malloc(sizeof(double) * (size_t)m1 * n1);
  double* Lc = (double*)malloc(sizeof(double) * (size_t)m1 * m1);
  double* Uc = (double*)malloc(sizeof(double) * (size_t)n1 * n1);
  int st = ORC_ERR_NOMEM;
  if (Xc && Lc && Uc) {
    for (int i = 0; i < m1; ++i)
      for (int j = 0; j < n1; ++j) Xc[(size_t)i * n1 + j] = X[(size_t)i * n + j];
    for (int i = 0; i < m1; ++i)
      for (int j = 0; j < m1; ++j) Lc[(size_t)i * m1 + j] = L[(size_t)i * m + j];
    for (int i = 0; i < n1; ++i)
      for (int j = 0; j < n1; ++j) Uc[(size_t)i * n1 + j] = U[(size_t)i * n + j];
    st = orc_round_nested(m1, n1, Xc, Lc, Uc, hint, tau, Z, Ypre, counts, hard_idx, hard_cap);
  }
  free(Xc);
  free(Lc);
  free(Uc);
  return st;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 3 (GPTQ-2D, Sec. 4.2) and Algorithm 6 (implicit Y, Appendix B)  */
/* ------------------------------------------------------------------------ */

int orc_round_gptq2d(int m, int n, const double* X, const double* L, const double* U,
                     const int32_t* hint, double tau, int32_t* Z, double* Ypre, int64_t* counts,
                     int64_t* hard_idx, int hard_cap) {
  double* Y = (double*)malloc(sizeof(double) * (size_t)m * n);
  double* C = (double*)calloc((size_t)m * n, sizeof(double));
  if (!Y || !C) { free(Y); free(C); return ORC_ERR_NOMEM; }
  memcpy(Y, X, sizeof(double) * (size_t)m * n);
  orc_replay rp;
  int64_t local[3];
  orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
  int bad = 0;
  /* 0-based anti-diagonal index s = i + j runs over 0 .. m+n-2 */
  for (int s = 0; s <= m + n - 2; ++s) {
    int ilo = s - (n - 1) > 0 ? s - (n - 1) : 0;
    int ihi = s < m - 1 ? s : m - 1;
    for (int i = ilo; i <= ihi; ++i) {
      int j = s - i;
      size_t o = (size_t)i * n + j;
      double y = Y[o];
      double z = orc_decide(y, o, &rp);
      double e = z - y;
      Z[o] = orc_to_int(z, &rp, &bad);
      Ypre[o] = y;
      for (int r = i; r < m; ++r) {
        double mm = L[(size_t)r * m + i] * e; /* M = L[:, i] E_ij */
        C[(size_t)r * n + j] += mm;           /* fold into C = L E */
        if (r > i) Y[(size_t)r * n + j] += mm; /* push down */
      }
    }
    for (int i = ilo; i <= ihi; ++i) {
      int j = s - i;
      double c = C[(size_t)i * n + j];
      for (int q = j + 1; q < n; ++q) Y[(size_t)i * n + q] += c * U[(size_t)j * n + q]; /* push right */
    }
  }
  free(Y);
  free(C);
  return bad ? ORC_ERR_RANGE : ORC_OK;
}

int orc_round_implicit(int m, int n, const double* X, const double* L, const double* U,
                       const int32_t* hint, double tau, int32_t* Z, double* Ypre,
                       int64_t* counts, int64_t* hard_idx, int hard_cap) {
  double* C = (double*)calloc((size_t)m * n, sizeof(double));
  double* Es = (double*)malloc(sizeof(double) * (size_t)(m < n ? n : m));
  if (!C || !Es) { free(C); free(Es); return ORC_ERR_NOMEM; }
  orc_replay rp;
  int64_t local[3];
  orc_replay_init(&rp, hint, tau, counts ? counts : local, hard_idx, hard_cap);
  int bad = 0;
  for (int s = 0; s <= m + n - 2; ++s) {
    int ilo = s - (n - 1) > 0 ? s - (n - 1) : 0;
    int ihi = s < m - 1 ? s : m - 1;
    for (int i = ilo; i <= ihi; ++i) {
      int j = s - i;
      size_t o = (size_t)i * n + j;
      double y = X[o]; /* Y_ij = X_ij + C[i, 0:j] U[0:j, j] (inclusive of j) */
      for (int q = 0; q <= j; ++q) y += C[(size_t)i * n + q] * U[(size_t)q * n + j];
      double z = orc_decide(y, o, &rp);
      Es[i] = z - y;
      Z[o] = orc_to_int(z, &rp, &bad);
      Ypre[o] = y;
    }
    for (int i = ilo; i <= ihi; ++i) {
      int j = s - i;
      for (int r = i; r < m; ++r) C[(size_t)r * n + j] += L[(size_t)r * m + i] * Es[i];
    }
  }
  free(C);
  free(Es);
  return bad ? ORC_ERR_RANGE : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Objective by definition (Eq. objective)                                   */
/* ------------------------------------------------------------------------ */

/* ||A (Z - X) B||_F^2 with extended-precision accumulation. */
double orc_objective(int m, int n, const double* X, const int32_t* Z, const double* A,
                     const double* B) {
  long double* T = (long double*)malloc(sizeof(long double) * (size_t)m * n);
  long double* rowsum = (long double*)malloc(sizeof(long double) * (size_t)m);
  double* R = (double*)malloc(sizeof(double) * (size_t)m * n);
  if (!T || !rowsum || !R) { free(T); free(rowsum); free(R); return NAN; }
  for (size_t k = 0; k < (size_t)m * n; ++k) R[k] = (double)Z[k] - X[k];
  /* T = A R */
#pragma omp parallel for schedule(static)
  for (int i = 0; i < m; ++i) {
    long double* t = T + (size_t)i * n;
    for (int j = 0; j < n; ++j) t[j] = 0.0L;
    for (int k = 0; k < m; ++k) {
      long double a = A[(size_t)i * m + k];
      if (a == 0.0L) continue;
      const double* r = R + (size_t)k * n;
      for (int j = 0; j < n; ++j) t[j] += a * r[j];
    }
  }
  /* sum over (i, j) of ((A R) B)_ij^2 */
#pragma omp parallel for schedule(static)
  for (int i = 0; i < m; ++i) {
    long double* v = (long double*)calloc((size_t)n, sizeof(long double));
    const long double* t = T + (size_t)i * n;
    for (int k = 0; k < n; ++k) {
      long double tk = t[k];
      if (tk == 0.0L) continue;
      const double* b = B + (size_t)k * n;
      for (int j = 0; j < n; ++j) v[j] += tk * b[j];
    }
    long double s = 0.0L;
    for (int j = 0; j < n; ++j) s += v[j] * v[j];
    rowsum[i] = s;
    free(v);
  }
  long double tot = 0.0L;
  for (int i = 0; i < m; ++i) tot += rowsum[i];
  free(T);
  free(rowsum);
  free(R);
  return (double)tot;
}

/* Number of OpenMP threads the oracle runs with (for reporting). */
int orc_num_threads(void) {
  int t = 1;
#ifdef _OPENMP
#pragma omp parallel
  {
#pragma omp single
    t = omp_get_num_threads();
  }
#endif
  return t;
}
