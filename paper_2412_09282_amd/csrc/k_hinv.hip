// Diagonal of the inverse of the damped Hessian proxy, the denominator of the W-A channel importance
// (Sec. 4.1 Eq. 7): [(H + delta I)^-1]_jj with H = X X^T and delta = damp * mean_j H_jj, in fp64.
//
// With the Cholesky factor L of A = H + delta I and T = L^-1 (lower triangular), A^-1 = T^T T, so
// [A^-1]_jj = sum_i T_ij^2: the squared norms of T's columns.  Both factors are formed by one blocked,
// right-looking sweep over 64-wide block columns k (the matrix padded to a multiple of 64 with an
// identity block, which leaves the leading part's inverse unchanged):
//   1. factor the diagonal block, A_kk = L_kk L_kk^T, and invert it, D_k = L_kk^-1   (one workgroup);
//   2. the panel L_ik = A_ik D_k^T (i > k) and T's block row k, T_kj = D_k B_kj (j <= k), whose
//      squared column sums are added to the result;
//   3. the trailing updates A_ij -= L_ik L_jk^T (k < j <= i) and B_ij -= L_ik T_kj (i > k, j <= k).
// B starts as the identity (block row i of B holds I - sum_{p < k} L_ip T_p at step k), so step 2
// is blocked forward substitution for T = L^-1, run alongside the factorization.  The 64 x 64 x 64
// products of steps 2 and 3 run on the fp64 matrix cores.  Only the lower triangle of H is read.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kHb = 64;  // block size
constexpr int kHs = 80;  // LDS stride of a k-major operand tile: 16 mod 32 doubles, so the two
                         // 16-lane halves of one operand read land in disjoint banks
typedef double d4v __attribute__((ext_vector_type(4)));

struct HinvWs {
  double* A;     // Np x Np: H + delta I, then the factor's off-diagonal blocks
  double* B;     // Np x Np: the forward-substitution right-hand sides, then T (lower blocks)
  double* D;     // nblk x 64 x 64: inverses of the diagonal blocks of L
  double* colsq; // Np: sum_i T_ij^2 so far
  double* prm;   // [0] delta
  int* flag;     // [0] nonzero once a pivot was not positive and finite
};

HinvWs carve_hinv(WsCursor& c, int64_t Np) {
  HinvWs w;
  w.A = c.take<double>(static_cast<size_t>(Np * Np));
  w.B = c.take<double>(static_cast<size_t>(Np * Np));
  w.D = c.take<double>(static_cast<size_t>(Np * kHb));
  w.colsq = c.take<double>(static_cast<size_t>(Np));
  w.prm = c.take<double>(4);
  w.flag = c.take<int>(4);
  return w;
}

// delta = damp * (sum_j H_jj) / N, summed in a fixed order; clears the flag.
__global__ __launch_bounds__(256) void hinv_delta_kernel(const double* __restrict__ H, int64_t ldh, int64_t N,
                                                         double damp, double* __restrict__ prm, int* __restrict__ flag) {
  __shared__ double s[256];
  const int tid = threadIdx.x;
  double a = 0.0;
  for (int64_t j = tid; j < N; j += 256) a += H[j * ldh + j];
  s[tid] = a;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) s[tid] += s[tid + h];
    __syncthreads();
  }
  if (tid == 0) {
    prm[0] = damp * (s[0] / static_cast<double>(N));
    flag[0] = 0;
  }
}

// A = H + delta I on the leading N x N (lower triangle read), identity on the padding; B = I on the
// lower blocks; the column sums cleared.
__global__ __launch_bounds__(256) void hinv_init_kernel(const double* __restrict__ H, int64_t ldh, int64_t N,
                                                        int64_t Np, const double* __restrict__ prm,
                                                        double* __restrict__ A, double* __restrict__ B,
                                                        double* __restrict__ colsq) {
  const double delta = prm[0];
  const int64_t total = Np * Np;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * 256) {
    if (e < Np) colsq[e] = 0.0;
    const int64_t i = e / Np, j = e - i * Np;
    if (j / kHb > i / kHb) continue;  // upper blocks are never read
    double a;
    if (i < N && j < N)
      a = (j <= i) ? H[i * ldh + j] + (i == j ? delta : 0.0) : 0.0;
    else
      a = (i == j) ? 1.0 : 0.0;
    A[e] = a;
    B[e] = (i == j) ? 1.0 : 0.0;
  }
}

// Step 1: Cholesky factor of the diagonal block k in LDS (column by column; the diagonal keeps the
// pivot until the end, since the trailing updates only read the scaled sub-diagonal column), then
// its inverse by forward substitution on the identity (row by row).  Writes D_k (zeros above the
// diagonal) and raises the flag on a pivot that is not positive and finite.
__global__ __launch_bounds__(256) void hinv_diag_kernel(const double* __restrict__ A, int64_t Np, int64_t k,
                                                        double* __restrict__ D, int* __restrict__ flag) {
  __shared__ double L[kHb][kHb + 1];
  __shared__ double T[kHb][kHb + 1];
  const int tid = threadIdx.x, col = tid & 63, rq = tid >> 6;
  const int64_t kb = k * kHb;
  for (int e = tid; e < kHb * kHb; e += 256) {
    const int r = e >> 6, c = e & 63;
    L[r][c] = (c <= r) ? A[(kb + r) * Np + kb + c] : 0.0;
    T[r][c] = (r == c) ? 1.0 : 0.0;
  }
  __syncthreads();
  bool bad = false;
  for (int c = 0; c < kHb; ++c) {
    if (tid < kHb && tid > c) {
      const double piv = L[c][c];
      L[tid][c] = L[tid][c] / sqrt(piv);
    }
    if (tid == 0) {
      const double piv = L[c][c];
      bad = bad || !(piv > 0.0 && piv < __builtin_inf());
    }
    __syncthreads();
    if (col > c) {
      const double ljc = L[col][c];
      for (int r = rq; r < kHb; r += 4)
        if (r >= col) L[r][col] -= L[r][c] * ljc;
    }
    __syncthreads();
  }
  if (tid < kHb) L[tid][tid] = sqrt(L[tid][tid]);
  __syncthreads();
  // T = L^-1: row p of T is final once divided by L_pp; it is then removed from the rows below.
  for (int p = 0; p < kHb; ++p) {
    if (tid < kHb) T[p][tid] = T[p][tid] / L[p][p];
    __syncthreads();
    {
      const double tp = T[p][col];
      for (int r = rq; r < kHb; r += 4)
        if (r > p) T[r][col] -= L[r][p] * tp;
    }
    __syncthreads();
  }
  for (int e = tid; e < kHb * kHb; e += 256) {
    const int r = e >> 6, c = e & 63;
    D[k * kHb * kHb + e] = (c <= r) ? T[r][c] : 0.0;
  }
  if (tid == 0 && bad) flag[0] = 1;
}

// dst[kk][r] = src[r * ld + kk]: a tile whose rows are the output index and columns the k index,
// stored k-major.  Lanes run over r, so the LDS writes are conflict-free.
__device__ __forceinline__ void load_t(double (*dst)[kHs], const double* __restrict__ src, int64_t ld, int tid) {
#pragma unroll 4
  for (int e = tid; e < kHb * kHb; e += 256) {
    const int r = e & 63, kk = e >> 6;
    dst[kk][r] = src[r * ld + kk];
  }
}
// dst[kk][j] = src[kk * ld + j]: a tile already k-major (coalesced).
__device__ __forceinline__ void load_d(double (*dst)[kHs], const double* __restrict__ src, int64_t ld, int tid) {
#pragma unroll 4
  for (int e = tid; e < kHb * kHb; e += 256) {
    const int j = e & 63, kk = e >> 6;
    dst[kk][j] = src[kk * ld + j];
  }
}

// acc = the 64 x 64 product of two k-major LDS tiles, one 32 x 32 quarter per wave as 2 x 2
// v_mfma_f64_16x16x4f64 tiles.  Lane l supplies A[i0 + l % 16][k + l / 16] and B[k + l / 16][j0 + l % 16]
// and holds C[i0 + l / 16 + 4 r][j0 + l % 16], r < 4.
__device__ __forceinline__ void mma64(const double (*Ak)[kHs], const double (*Bk)[kHs], d4v (&acc)[2][2], int wi,
                                      int wj, int li, int lk) {
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = d4v{0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int ks = 0; ks < kHb; ks += 4) {
    const double a0 = Ak[ks + lk][wi + li], a1 = Ak[ks + lk][wi + 16 + li];
    const double b0 = Bk[ks + lk][wj + li], b1 = Bk[ks + lk][wj + 16 + li];
    acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
  }
}

// Step 2.  Workgroups below nbelow: L_ik = A_ik D_k^T for block row i = k + 1 + g (in place in A).
// The others: T_kj = D_k B_kj for block column j = g - nbelow <= k (in place in B), and the squared
// column sums of T_kj (rows in order) added to colsq.
__global__ __launch_bounds__(256) void hinv_panel_kernel(double* __restrict__ A, double* __restrict__ B, int64_t Np,
                                                         int64_t k, int64_t nbelow, const double* __restrict__ D,
                                                         double* __restrict__ colsq) {
  __shared__ double Ak[kHb][kHs];
  __shared__ double Bk[kHb][kHs];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32, li = lane & 15, lk = lane >> 4;
  const int64_t g = blockIdx.x, kb = k * kHb;
  const double* Dk = D + k * kHb * kHb;
  const bool lpart = g < nbelow;
  double* C;
  if (lpart) {
    const int64_t ib = (k + 1 + g) * kHb;
    C = A + ib * Np + kb;
    load_t(Ak, C, Np, tid);
    load_t(Bk, Dk, kHb, tid);
  } else {
    const int64_t jb = (g - nbelow) * kHb;
    C = B + kb * Np + jb;
    load_t(Ak, Dk, kHb, tid);
    load_d(Bk, C, Np, tid);
  }
  __syncthreads();
  d4v acc[2][2];
  mma64(Ak, Bk, acc, wi, wj, li, lk);
  if (lpart) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) C[(wi + 16 * a + lk + 4 * r) * Np + wj + 16 * b + li] = acc[a][b][r];
    return;
  }
  // T_kj: through LDS (the operand tiles are no longer read), written row-major, then column sums
  __syncthreads();
  double (*Ts)[kHs] = Ak;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) Ts[wi + 16 * a + lk + 4 * r][wj + 16 * b + li] = acc[a][b][r];
  __syncthreads();
  for (int e = tid; e < kHb * kHb; e += 256) {
    const int r = e >> 6, c = e & 63;
    C[r * Np + c] = Ts[r][c];
  }
  if (tid < kHb) {
    double s = 0.0;
    for (int r = 0; r < kHb; ++r) s += Ts[r][tid] * Ts[r][tid];
    colsq[(g - nbelow) * kHb + tid] += s;
  }
}

// Step 3.  Workgroups below ntri: the lower-triangle tiles (a >= b) of the trailing matrix,
// A_ij -= L_ik L_jk^T with i = k + 1 + a, j = k + 1 + b.  The others: B_ij -= L_ik T_kj for
// i = k + 1 + a, j <= k.
__global__ __launch_bounds__(256) void hinv_update_kernel(double* __restrict__ A, double* __restrict__ B, int64_t Np,
                                                          int64_t k, int64_t ntri) {
  __shared__ double Ak[kHb][kHs];
  __shared__ double Bk[kHb][kHs];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32, li = lane & 15, lk = lane >> 4;
  const int64_t g = blockIdx.x, kb = k * kHb;
  double* C;
  if (g < ntri) {
    // g = a (a + 1) / 2 + b, 0 <= b <= a
    int64_t a = static_cast<int64_t>((sqrt(8.0 * static_cast<double>(g) + 1.0) - 1.0) * 0.5);
    while (a * (a + 1) / 2 > g) --a;
    while ((a + 1) * (a + 2) / 2 <= g) ++a;
    const int64_t b = g - a * (a + 1) / 2;
    const int64_t ib = (k + 1 + a) * kHb, jb = (k + 1 + b) * kHb;
    load_t(Ak, A + ib * Np + kb, Np, tid);
    load_t(Bk, A + jb * Np + kb, Np, tid);
    C = A + ib * Np + jb;
  } else {
    const int64_t h = g - ntri, a = h / (k + 1), j = h - a * (k + 1);
    const int64_t ib = (k + 1 + a) * kHb, jb = j * kHb;
    load_t(Ak, A + ib * Np + kb, Np, tid);
    load_d(Bk, B + kb * Np + jb, Np, tid);
    C = B + ib * Np + jb;
  }
  __syncthreads();
  d4v acc[2][2];
  mma64(Ak, Bk, acc, wi, wj, li, lk);
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        double* p = C + (wi + 16 * a + lk + 4 * r) * Np + wj + 16 * b + li;
        *p = *p - acc[a][b][r];
      }
}

// hinv[j] = colsq[j] and scale[j] = float(1 / (2 colsq[j])), or NaN for all when the flag is set.
__global__ __launch_bounds__(256) void hinv_finish_kernel(int64_t N, const double* __restrict__ colsq,
                                                          const int* __restrict__ flag, double* __restrict__ hinv,
                                                          float* __restrict__ scale) {
  const bool bad = flag[0] != 0;
  for (int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; j < N;
       j += static_cast<int64_t>(gridDim.x) * 256) {
    const double v = bad ? __builtin_nan("") : colsq[j];
    if (hinv) hinv[j] = v;
    if (scale) scale[j] = static_cast<float>(1.0 / (2.0 * v));
  }
}

}  // namespace

size_t hinv_ws_bytes(int64_t N) {
  const int64_t Np = (N + kHb - 1) / kHb * kHb;
  WsCursor c(nullptr);
  (void)carve_hinv(c, Np);
  return c.used;
}

hipError_t launch_hinv(const double* H, int64_t ldh, int64_t N, double damp, double* hinv, float* scale, void* ws,
                       hipStream_t stream) {
  const int64_t nblk = (N + kHb - 1) / kHb, Np = nblk * kHb;
  WsCursor c(ws);
  const HinvWs w = carve_hinv(c, Np);
  hipLaunchKernelGGL(hinv_delta_kernel, dim3(1), dim3(256), 0, stream, H, ldh, N, damp, w.prm, w.flag);
  const int64_t ig = std::min<int64_t>(cdiv(Np * Np, 256), 65536);
  hipLaunchKernelGGL(hinv_init_kernel, dim3(static_cast<unsigned>(ig)), dim3(256), 0, stream, H, ldh, N, Np, w.prm,
                     w.A, w.B, w.colsq);
  for (int64_t k = 0; k < nblk; ++k) {
    hipLaunchKernelGGL(hinv_diag_kernel, dim3(1), dim3(256), 0, stream, w.A, Np, k, w.D, w.flag);
    const int64_t nbelow = nblk - 1 - k;
    hipLaunchKernelGGL(hinv_panel_kernel, dim3(static_cast<unsigned>(nbelow + k + 1)), dim3(256), 0, stream, w.A, w.B,
                       Np, k, nbelow, w.D, w.colsq);
    if (nbelow > 0) {
      const int64_t ntri = nbelow * (nbelow + 1) / 2, nrect = nbelow * (k + 1);
      hipLaunchKernelGGL(hinv_update_kernel, dim3(static_cast<unsigned>(ntri + nrect)), dim3(256), 0, stream, w.A,
                         w.B, Np, k, ntri);
    }
  }
  hipLaunchKernelGGL(hinv_finish_kernel, dim3(static_cast<unsigned>(std::min<int64_t>(cdiv(N, 256), 4096))),
                     dim3(256), 0, stream, N, w.colsq, w.flag, hinv, scale);
  return hipGetLastError();
}

}  // namespace crvq
