// Column (input-channel) reduction behind CRVQ's channel importance (Sec. 4.1 Eq. 7, Appendix A.2
// Eq. 9-10 of the paper) and the Hessian diagonal [X X^T]_jj:
//   out[j] = s_j * R_i (A[i,j] - B[i,j])^2,  R = sum (fp64) or max.
// Pass 1: threads own 4 adjacent columns (16-byte fp32 / 8-byte bf16 loads, so every row of a
// wave is one contiguous 1 KiB / 512 B segment); the grid's second dimension splits the rows into
// slabs that each write an fp64 partial per column.  Pass 2 folds the slabs in slab order and
// applies the scale.  Both passes are deterministic.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kCols = 4;          // columns per thread
#ifndef CRVQ_CR_ROWS
#define CRVQ_CR_ROWS 8
#endif
constexpr int kRowsInFlight = CRVQ_CR_ROWS;  // row loads issued back to back per thread

// kCols elements of one row as floats: one 16-byte (fp32) or 8-byte (bf16) load when the columns
// are full and aligned, element loads otherwise; zero past the last column.
template <int TY>
__device__ __forceinline__ void load4f(const void* p, int64_t idx, int valid_cols, float (&v)[kCols]) {
  if constexpr (TY == ET_F32) {
    const float* f = static_cast<const float*>(p) + idx;
    if (valid_cols == kCols && ((reinterpret_cast<uintptr_t>(f) & 15) == 0)) {
      const uint4 q = ld_stream(f);
      v[0] = __uint_as_float(q.x);
      v[1] = __uint_as_float(q.y);
      v[2] = __uint_as_float(q.z);
      v[3] = __uint_as_float(q.w);
    } else {
#pragma unroll
      for (int c = 0; c < kCols; ++c) v[c] = (c < valid_cols) ? f[c] : 0.0f;
    }
  } else {
    const uint16_t* h = static_cast<const uint16_t*>(p) + idx;
    if (valid_cols == kCols && ((reinterpret_cast<uintptr_t>(h) & 7) == 0)) {
      const uint2 q = ld_stream8(h);
      v[0] = __uint_as_float(q.x << 16);
      v[1] = __uint_as_float(q.x & 0xffff0000u);
      v[2] = __uint_as_float(q.y << 16);
      v[3] = __uint_as_float(q.y & 0xffff0000u);
    } else {
#pragma unroll
      for (int c = 0; c < kCols; ++c)
        v[c] = (c < valid_cols) ? __uint_as_float(static_cast<uint32_t>(h[c]) << 16) : 0.0f;
    }
  }
}

// Pass 1 of one (input type, B present, reduction) combination.  The raw row values stay floats
// while in flight (fewer registers, more waves); each is widened to fp64 when it is accumulated:
// x = a - b in fp64, x * x in fp64, then the fp64 sum or max, rows in ascending order.
template <int TY, bool HAS_B, bool MAX>
__global__ __launch_bounds__(256) void colreduce_partial(const void* __restrict__ A, int64_t lda,
                                                         const void* __restrict__ B, int64_t ldb, int64_t M,
                                                         int64_t N, int64_t rows_per_slab, double* __restrict__ part) {
  const int64_t j0 = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * kCols;
  if (j0 >= N) return;
  const int valid_cols = static_cast<int>((N - j0) < kCols ? (N - j0) : kCols);
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * rows_per_slab;
  const int64_t i1 = (i0 + rows_per_slab < M) ? i0 + rows_per_slab : M;
  double acc[kCols] = {0.0, 0.0, 0.0, 0.0};
  auto fold = [&](const float (&a)[kCols], const float (&b)[kCols]) {
#pragma unroll
    for (int c = 0; c < kCols; ++c) {
      const double x = HAS_B ? static_cast<double>(a[c]) - static_cast<double>(b[c]) : static_cast<double>(a[c]);
      const double sq = x * x;
      acc[c] = MAX ? (sq > acc[c] ? sq : acc[c]) : acc[c] + sq;
    }
  };
  int64_t i = i0;
  for (; i + kRowsInFlight <= i1; i += kRowsInFlight) {
    float a[kRowsInFlight][kCols], b[kRowsInFlight][kCols];
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) load4f<TY>(A, (i + u) * lda + j0, valid_cols, a[u]);
    if constexpr (HAS_B) {
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) load4f<TY>(B, (i + u) * ldb + j0, valid_cols, b[u]);
    }
#pragma unroll
    for (int u = 0; u < kRowsInFlight; ++u) fold(a[u], b[u]);
  }
  for (; i < i1; ++i) {
    float a[kCols], b[kCols];
    load4f<TY>(A, i * lda + j0, valid_cols, a);
    if constexpr (HAS_B) load4f<TY>(B, i * ldb + j0, valid_cols, b);
    fold(a, b);
  }
#pragma unroll
  for (int c = 0; c < kCols; ++c)
    if (c < valid_cols) part[static_cast<int64_t>(blockIdx.y) * N + j0 + c] = acc[c];
}

// Block of 256 threads per 64 columns: thread (column c, lane group q) folds slabs q, q + 4, ... in
// order, then the four group sums are combined in group order.
__global__ __launch_bounds__(256) void colreduce_final(const double* __restrict__ part, int slabs, int64_t N,
                                                       const float* __restrict__ scale, int reduce,
                                                       float* __restrict__ out) {
  __shared__ double sh[4][64];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 64 + c;
  double acc = 0.0;
  if (j < N) {
#pragma unroll 4
    for (int s = q; s < slabs; s += 4) {
      const double v = part[static_cast<int64_t>(s) * N + j];
      acc = (reduce == 0) ? acc + v : (v > acc ? v : acc);
    }
  }
  sh[q][c] = acc;
  __syncthreads();
  if (q == 0 && j < N) {
    double r = sh[0][c];
    for (int g = 1; g < 4; ++g) r = (reduce == 0) ? r + sh[g][c] : (sh[g][c] > r ? sh[g][c] : r);
    out[j] = static_cast<float>(scale ? static_cast<double>(scale[j]) * r : r);
  }
}

struct Plan {
  int64_t col_blocks;
  int64_t slabs;
  int64_t rows_per_slab;
};

Plan plan(int64_t M, int64_t N) {
  Plan p;
  p.col_blocks = cdiv(cdiv(N, kCols), 256);
  int64_t want = cdiv(4096, p.col_blocks);      // aim for >= 4096 blocks in flight
  if (want > 512) want = 512;                   // bounds the fp64 partials (slabs x N)
  int64_t max_slabs = cdiv(M, 16);              // at least 16 rows per slab
  p.slabs = want < max_slabs ? want : max_slabs;
  if (p.slabs < 1) p.slabs = 1;
  p.rows_per_slab = cdiv(M, p.slabs);
  p.slabs = cdiv(M, p.rows_per_slab);
  return p;
}

}  // namespace

size_t colreduce_ws_bytes(int64_t M, int64_t N) {
  Plan p = plan(M, N);
  return align256(static_cast<size_t>(p.slabs * N) * sizeof(double));
}

hipError_t launch_colreduce(const void* A, int64_t lda, const void* B, int64_t ldb, int type, int64_t M, int64_t N,
                            const float* scale, int reduce, float* out, void* ws, hipStream_t stream) {
  Plan p = plan(M, N);
  double* part = static_cast<double*>(ws);
  const dim3 grid(static_cast<unsigned>(p.col_blocks), static_cast<unsigned>(p.slabs));
  const int combo = (type == ET_BF16 ? 4 : 0) + (B ? 2 : 0) + (reduce != 0 ? 1 : 0);
  switch (combo) {
#define CRVQ_COLRED(CASE, TY, HB, MX)                                                                        \
  case CASE:                                                                                                 \
    hipLaunchKernelGGL((colreduce_partial<TY, HB, MX>), grid, dim3(256), 0, stream, A, lda, B, ldb, M, N, \
                       p.rows_per_slab, part);                                                               \
    break;
    CRVQ_COLRED(0, ET_F32, false, false)
    CRVQ_COLRED(1, ET_F32, false, true)
    CRVQ_COLRED(2, ET_F32, true, false)
    CRVQ_COLRED(3, ET_F32, true, true)
    CRVQ_COLRED(4, ET_BF16, false, false)
    CRVQ_COLRED(5, ET_BF16, false, true)
    CRVQ_COLRED(6, ET_BF16, true, false)
    CRVQ_COLRED(7, ET_BF16, true, true)
#undef CRVQ_COLRED
  }
  hipLaunchKernelGGL(colreduce_final, dim3(static_cast<unsigned>(cdiv(N, 64))), dim3(256), 0, stream, part,
                     static_cast<int>(p.slabs), N, scale, reduce, out);
  return hipGetLastError();
}

}  // namespace crvq
