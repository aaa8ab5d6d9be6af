// Device building blocks shared by the factorisation and the sweep kernels.
//
// Everything works on 64 x 64 tiles of fp64 data with one 256-thread
// workgroup (four wave64s) per tile. Dense contractions go through
// v_mfma_f64_16x16x4f64. Lane layout of that instruction on gfx950 (checked on
// the device with an in-bounds probe):
//   A (16 x 4): lane l holds A[l % 16][l / 16]
//   B (4 x 16): lane l holds B[l / 16][l % 16]
//   D (16 x 16): element r (0..3) of lane l is D[4 r + l / 16][l % 16]
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace g2d {

constexpr int TB = 64;     // tile edge (rows and columns)
constexpr int NT = 256;    // threads per workgroup
constexpr int KC = 16;     // contraction chunk staged through LDS
constexpr int SA = TB + 2; // LDS row stride (doubles) of a staged chunk

typedef double d4 __attribute__((ext_vector_type(4)));

// k-major staging buffers of one contraction chunk: a[k][row], b[k][col].
struct GemmSmem {
  double a[KC][SA];
  double b[KC][SA];
};

// Accumulator of one 64 x 64 output tile. Wave w owns rows 32*(w>>1) .. +32
// and columns 32*(w&1) .. +32 as four 16 x 16 MFMA blocks t[2u+v]; element r
// of lane l in block (u, v) is tile entry
//   row = 32*(w>>1) + 16u + 4r + (l>>4),  col = 32*(w&1) + 16v + (l&15).
struct Acc {
  d4 t[4];
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = d4{0.0, 0.0, 0.0, 0.0};
  }
};

__device__ __forceinline__ int acc_row(int u, int r) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  return 32 * (w >> 1) + 16 * u + 4 * r + (l >> 4);
}
__device__ __forceinline__ int acc_col(int v) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  return 32 * (w & 1) + 16 * v + (l & 15);
}

// ---------------------------------------------------------------------------
// Operand fetchers. An operand is a 64-wide index i (rows of the left factor,
// columns of the right factor) times the contraction index k. Each thread
// fetches four values of a 16-deep chunk into registers (so the next chunk's
// global loads overlap the current chunk's MFMAs) and then puts them into the
// k-major LDS buffer.
// ---------------------------------------------------------------------------

// element (i, k) at p[i*ld + k] (i-rows contiguous along k); fp64, in bounds,
// p and ld 32-byte aligned.
struct OpRK {
  const double* p;
  int64_t ld;
  __device__ __forceinline__ void fetch(int k0, double v[4]) const {
    const int t = threadIdx.x;
    const double2* q = reinterpret_cast<const double2*>(p + (int64_t)(t >> 2) * ld + k0 + (t & 3) * 4);
    double2 x = q[0], y = q[1];
    v[0] = x.x; v[1] = x.y; v[2] = y.x; v[3] = y.y;
  }
  __device__ __forceinline__ static void put(double (*s)[SA], const double v[4]) {
    const int t = threadIdx.x, i = t >> 2, kq = (t & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) s[kq + e][i] = v[e];
  }
};

// element (i, k) at p[k*ld + i] (k-rows contiguous along i); fp64, in bounds.
struct OpKR {
  const double* p;
  int64_t ld;
  __device__ __forceinline__ void fetch(int k0, double v[4]) const {
    const int t = threadIdx.x;
    const double2* q = reinterpret_cast<const double2*>(p + (int64_t)(k0 + (t >> 4)) * ld + (t & 15) * 4);
    double2 x = q[0], y = q[1];
    v[0] = x.x; v[1] = x.y; v[2] = y.x; v[3] = y.y;
  }
  __device__ __forceinline__ static void put(double (*s)[SA], const double v[4]) {
    const int t = threadIdx.x, k = t >> 4, iq = (t & 15) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) s[k][iq + e] = v[e];
  }
};

// Four MFMA k-steps over one staged chunk.
__device__ __forceinline__ void mma_chunk(Acc& acc, const GemmSmem& sm) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int rb = 32 * (w >> 1) + (l & 15), cb = 32 * (w & 1) + (l & 15);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int k = 4 * kk + (l >> 4);
    const double a0 = sm.a[k][rb], a1 = sm.a[k][rb + 16];
    const double b0 = sm.b[k][cb], b1 = sm.b[k][cb + 16];
    acc.t[0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc.t[0], 0, 0, 0);
    acc.t[1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc.t[1], 0, 0, 0);
    acc.t[2] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc.t[2], 0, 0, 0);
    acc.t[3] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc.t[3], 0, 0, 0);
  }
}

// acc += opA (64 x K) * opB (K x 64), K a multiple of 16. All 256 threads of
// the workgroup must call it; it starts and ends with a barrier-safe state.
template <class OA, class OB>
__device__ void gemm_acc(Acc& acc, const OA& oa, const OB& ob, int K, GemmSmem& sm) {
  if (K <= 0) return;
  double va[4], vb[4];
  oa.fetch(0, va);
  ob.fetch(0, vb);
  for (int k0 = 0; k0 < K; k0 += KC) {
    __syncthreads();
    OA::put(sm.a, va);
    OB::put(sm.b, vb);
    __syncthreads();
    if (k0 + KC < K) {
      oa.fetch(k0 + KC, va);
      ob.fetch(k0 + KC, vb);
    }
    mma_chunk(acc, sm);
  }
  __syncthreads();
}

// acc (+)= C tile at p (row-major, ld).
__device__ __forceinline__ void acc_add_from(Acc& acc, const double* p, int64_t ld) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc.t[2 * u + v][r] += p[(int64_t)acc_row(u, r) * ld + acc_col(v)];
}

__device__ __forceinline__ void acc_store(const Acc& acc, double* p, int64_t ld, double scale) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) p[(int64_t)acc_row(u, r) * ld + acc_col(v)] = scale * acc.t[2 * u + v][r];
}

// Writes the accumulator tile into an LDS array s[64][ld].
template <int LD>
__device__ __forceinline__ void acc_to_lds(const Acc& acc, double (*s)[LD]) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r) s[acc_row(u, r)][acc_col(v)] = acc.t[2 * u + v][r];
}


// ---------------------------------------------------------------------------
// Whole-block staging: both operands of a 64-deep contraction are loaded into
// registers at once (one memory latency), written k-major into LDS and
// consumed by 64 MFMA k-steps per wave.
// ---------------------------------------------------------------------------

// A whole 64-deep contraction block of both operands, k-major.
constexpr int GSA = TB + 1;  // odd stride: transposed writes spread over the banks
constexpr int GSB = TB + 2;
struct Stage64 {
  double a[TB][GSA];  // a[k][i] = A[i][k]
  double b[TB][GSB];  // b[k][j] = B[k][j]
};

// 64 x 64 fp64 block at p (row-major, ld) into registers: element
// (e >> 6, e & 63) with e = threadIdx.x + 256 s goes to r[s] (coalesced).
__device__ __forceinline__ void load_blk(const double* p, int64_t ld, double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    r[s] = p[(int64_t)(e >> 6) * ld + (e & 63)];
  }
}
// left operand A[i][k] = r -> a[k][i]
__device__ __forceinline__ void put_a(Stage64& st, const double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    st.a[e & 63][e >> 6] = r[s];
  }
}
// right operand B[k][j] = r -> b[k][j]
__device__ __forceinline__ void put_b(Stage64& st, const double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    st.b[e >> 6][e & 63] = r[s];
  }
}
// acc += (staged A) (staged B) over the 64-deep block.
__device__ __forceinline__ void mma_blk(Acc& acc, const Stage64& st) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int rb = 32 * (w >> 1) + (l & 15), cb = 32 * (w & 1) + (l & 15);
#pragma unroll
  for (int kk = 0; kk < TB / 4; ++kk) {
    const int k = 4 * kk + (l >> 4);
    const double a0 = st.a[k][rb], a1 = st.a[k][rb + 16];
    const double b0 = st.b[k][cb], b1 = st.b[k][cb + 16];
    acc.t[0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc.t[0], 0, 0, 0);
    acc.t[1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc.t[1], 0, 0, 0);
    acc.t[2] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc.t[2], 0, 0, 0);
    acc.t[3] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc.t[3], 0, 0, 0);
  }
}

// right operand given transposed, B^T[j][k] = r -> b[k][j]
__device__ __forceinline__ void put_bt(Stage64& st, const double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    st.b[e & 63][e >> 6] = r[s];
  }
}

// ---------------------------------------------------------------------------
// Tile-contiguous storage of the factors and the sweep's matrices. A padded
// matrix with TC tile columns is stored tile by tile: tile (I, J) occupies the
// 4096 doubles from (I TC + J) 4096 on, in one of two orders:
//   R (row-major tile): entry (r, c) at r 64 + c           (U, E, P, R)
//   S (split tile): the two 64 x 32 column halves one after the other, each
//     row-major: entry (r, c) at (c / 32) 2048 + r 32 + c % 32   (L, C)
// L and C are the left operands of the deferred-feedback products, read in
// 32-deep chunks: in S order four rows of a chunk are 1 KB of contiguous
// memory, and in either order a chunk of a tile is 16 KB of it.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ int64_t tile_off(int I, int J, int TC) {
  return ((int64_t)I * TC + J) << 12;
}
__host__ __device__ __forceinline__ int r_idx(int r, int c) { return (r << 6) + c; }
__host__ __device__ __forceinline__ int s_idx(int r, int c) { return ((c >> 5) << 11) + (r << 5) + (c & 31); }
// entry (i, j) of a matrix with TC tile columns
__host__ __device__ __forceinline__ int64_t r_at(int64_t i, int64_t j, int TC) {
  return tile_off((int)(i >> 6), (int)(j >> 6), TC) + r_idx((int)(i & 63), (int)(j & 63));
}
__host__ __device__ __forceinline__ int64_t s_at(int64_t i, int64_t j, int TC) {
  return tile_off((int)(i >> 6), (int)(j >> 6), TC) + s_idx((int)(i & 63), (int)(j & 63));
}

// 64 x 64 tile in S order into registers, in load_blk's element order.
__device__ __forceinline__ void load_blk_s(const double* p, double r[16]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const int e = t + NT * s;
    r[s] = p[s_idx(e >> 6, e & 63)];
  }
}

// Device-scope error flags (bit set with a relaxed atomic OR).
enum : int { FLAG_SINGULAR = 1, FLAG_NONFINITE = 2, FLAG_OVERFLOW = 4, FLAG_TIMEOUT = 8 };

__device__ __forceinline__ void raise_flag(int* flags, int bit) {
  __hip_atomic_fetch_or(flags, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace g2d
