// Diagonal of the inverse of the damped Hessian proxy, the denominator of the W-A channel importance
// (Sec. 4.1 Eq. 7): [(H + delta I)^-1]_jj with H = X X^T and delta = damp * mean_j H_jj, in fp64.
//
// With the Cholesky factor L of A = H + delta I and T = L^-1 (lower triangular), A^-1 = T^T T, so
// [A^-1]_jj = sum_i T_ij^2: the squared norms of T's columns.  Both factors are formed by one blocked,
// right-looking sweep over 64-wide block columns k (the matrix padded to a multiple of 64 with an
// identity block, which leaves the leading part's inverse unchanged):
//   1. factor the diagonal block, A_kk = L_kk L_kk^T, and invert it, D_k = L_kk^-1;
//   2. the panel L_ik = A_ik D_k^T (i > k) and T's block row k, T_kj = D_k B_kj (j <= k), whose
//      squared column sums are added to the result (steps 1 and 2 are one launch);
//   3. the trailing updates A_ij -= L_ik L_jk^T (k < j <= i) and B_ij -= L_ik T_kj (i > k, j <= k).
// B starts as the identity (block row i of B holds I - sum_{p < k} L_ip T_p at step k), so step 2
// is blocked forward substitution for T = L^-1, run alongside the factorization.  The 64 x 64 x 64
// products of steps 2 and 3 run on the fp64 matrix cores.  Only the lower triangle of H is read.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kHb = 64;  // block size
constexpr int kHr = 66;  // LDS stride of a row-major operand tile (element (row, k) at [row][k]): 2 mod 32
                         // doubles, so an MFMA operand read (16 rows x 2 k per half wave) is conflict-free
constexpr int kHs = 80;  // LDS stride of a k-major operand tile (element (k, col) at [k][col]): 16 mod 32
typedef double d4v __attribute__((ext_vector_type(4)));
typedef double d2v __attribute__((ext_vector_type(2)));

struct HinvWs {
  double* A;     // Np x Np: H + delta I, then the factor's off-diagonal blocks
  double* B;     // Np x Np: the forward-substitution right-hand sides, then T (lower blocks)
  double* colsq; // Np: sum_i T_ij^2 so far
  double* prm;   // [0] delta
  int* flag;     // [0] nonzero once a pivot was not positive and finite
};

HinvWs carve_hinv(WsCursor& c, int64_t Np) {
  HinvWs w;
  w.A = c.take<double>(static_cast<size_t>(Np * Np));
  w.B = c.take<double>(static_cast<size_t>(Np * Np));
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

// 1 / sqrt(x) for x > 0: the hardware estimate refined by three Newton steps (each squares the
// relative error; the estimate is good to about 2^-22), a few ulps from the rounded quotient.  Not
// positive or not finite x gives NaN or 0, which the caller's pivot check has already flagged.
__device__ __forceinline__ double rsqrt_f64(double x) {
  double y = __builtin_amdgcn_rsq(x);
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const double h = x * y;                       // ~ sqrt(x)
    const double e = __builtin_fma(-h, y, 1.0);   // 1 - x y^2
    y = __builtin_fma(0.5 * y, e, y);
  }
  return y;
}

// dst[r][k] = src[r * ld + k] for a 64 x 64 tile (row-major in LDS, stride kHr), 16-byte loads, each
// wave reading two whole rows per instruction.
__device__ __forceinline__ void load_rows(double (*dst)[kHr], const double* __restrict__ src, int64_t ld, int tid) {
#pragma unroll
  for (int e = tid; e < kHb * kHb / 2; e += 256) {
    const int r = e >> 5, m = (e & 31) * 2;
    const d2v v = *reinterpret_cast<const d2v*>(src + r * ld + m);
    *reinterpret_cast<d2v*>(&dst[r][m]) = v;
  }
}
// dst[k][j] = src[k * ld + j] (k-major in LDS, stride kHs).
__device__ __forceinline__ void load_kmaj(double (*dst)[kHs], const double* __restrict__ src, int64_t ld, int tid) {
#pragma unroll
  for (int e = tid; e < kHb * kHb / 2; e += 256) {
    const int k = e >> 5, m = (e & 31) * 2;
    const d2v v = *reinterpret_cast<const d2v*>(src + k * ld + m);
    *reinterpret_cast<d2v*>(&dst[k][m]) = v;
  }
}

// acc = A B for 64 x 64 tiles, one 32 x 32 quarter per wave as 2 x 2 v_mfma_f64_16x16x4f64 tiles.
// A is row-major (element (i, k) at Ar[i][k]); B is given either as the rows of B^T (element (k, j)
// at Br[j][k], BT = true) or k-major (at Bk[k][j]).  Lane l supplies A[i0 + l % 16][k + l / 16] and
// B[k + l / 16][j0 + l % 16] and holds C[i0 + l / 16 + 4 r][j0 + l % 16], r < 4.
template <bool BT>
__device__ __forceinline__ void mma64(const double (*Ar)[kHr], const double* Bs, d4v (&acc)[2][2], int wi, int wj,
                                      int li, int lk) {
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = d4v{0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int ks = 0; ks < kHb; ks += 4) {
    const double a0 = Ar[wi + li][ks + lk], a1 = Ar[wi + 16 + li][ks + lk];
    double b0, b1;
    if (BT) {
      b0 = Bs[(wj + li) * kHr + ks + lk];
      b1 = Bs[(wj + 16 + li) * kHr + ks + lk];
    } else {
      b0 = Bs[(ks + lk) * kHs + wj + li];
      b1 = Bs[(ks + lk) * kHs + wj + 16 + li];
    }
    acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
  }
}

// Steps 1 and 2 of block column k in one launch.  Every workgroup first factors the diagonal block
// itself (the factorization is a latency chain, so repeating it costs no time and saves a launch and
// a round trip through memory) and forms D_k = L_kk^-1; then workgroups g < nbelow form the panel
// L_ik = A_ik D_k^T of block row i = k + 1 + g (in place in A), the others T's block T_kj = D_k B_kj of
// block column j = g - nbelow <= k (in place in B) and add its squared column sums (rows in order).
//
// The factorization: thread (rq, col) = (wave, lane) holds rows rq + 4 q (q < 16) of column col of
// the block for L and for T (T starts as I).  At step c the owners of column c scale it by
// 1 / sqrt(pivot) and the owners of row c of T divide it by the same square root, both publishing
// through LDS; then every thread removes column c from its trailing elements of L (Cholesky) and
// row c of T from its rows below c (forward substitution on the identity).  Two barriers per step.
// The diagonal of L is never stored: the scaled column and T only need 1 / sqrt(pivot).
__global__ __launch_bounds__(256) void hinv_step_kernel(double* __restrict__ A, double* __restrict__ B, int64_t Np,
                                                        int64_t k, int64_t nbelow, double* __restrict__ colsq,
                                                        int* __restrict__ flag) {
  __shared__ double Dr[kHb][kHr];  // D_k, row-major
  __shared__ double Or[kHb][kHr];  // the other operand: A_ik rows, or T_kj through LDS at the end
  __shared__ double Ok[kHb][kHs];  // B_kj, k-major
  __shared__ double colbuf[4][16];
  __shared__ double rowbuf[kHb];
  __shared__ double prow[kHb];  // row c of the partly reduced block: prow[c] is the next pivot
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane, rq = wave;
  const int64_t g = blockIdx.x, kb = k * kHb;
  const bool lpart = g < nbelow;
  // this workgroup's operand tile, in flight during the factorization
  double* C;
  if (lpart) {
    C = A + ((k + 1 + g) * kHb) * Np + kb;
    load_rows(Or, C, Np, tid);
  } else {
    C = B + kb * Np + (g - nbelow) * kHb;
    load_kmaj(Ok, C, Np, tid);
  }
  // rq is the wave index, uniform in the wave (readfirstlane tells the compiler), so every test on a
  // row r = rq + 4 q below is a scalar branch
  const int rqs = __builtin_amdgcn_readfirstlane(rq);
  double aL[16], aT[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int r = rqs + 4 * q;
    aL[q] = (col <= r) ? A[(kb + r) * Np + kb + col] : 0.0;
    aT[q] = (col == r) ? 1.0 : 0.0;
  }
  if (rqs == 0) prow[col] = aL[0];
  __syncthreads();
  bool bad = false;
  for (int c = 0; c < kHb; ++c) {
    const double piv = prow[c];
    const double inv_d = rsqrt_f64(piv);
    bad = bad || !(piv > 0.0 && piv < __builtin_inf());
    if (col == c) {
      // column c of L below the diagonal (the diagonal itself is not needed again)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int r = rqs + 4 * q;
        if (r > c) aL[q] *= inv_d;
        colbuf[rqs][q] = (r > c) ? aL[q] : 0.0;
      }
    }
    if (rqs == (c & 3)) {
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (q == (c >> 2)) {
          aT[q] *= inv_d;
          rowbuf[col] = aT[q];
        }
    }
    __syncthreads();
    double cb[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) cb[q] = colbuf[rqs][q];
    // L[col][c] (zero unless col > c) and T[c][col].  The products below vanish wherever the update
    // does not apply (rows r <= c have cb = 0; columns col <= c have ljc = 0), so they run unmasked;
    // elements above the diagonal of L collect values that are never read.
    const double ljc = colbuf[col & 3][col >> 2], tc = rowbuf[col];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      aL[q] = __builtin_fma(-cb[q], ljc, aL[q]);
      aT[q] = __builtin_fma(-cb[q], tc, aT[q]);
    }
    if (rqs == ((c + 1) & 3)) {
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (q == ((c + 1) >> 2)) prow[col] = aL[q];
    }
    __syncthreads();
  }
  if (g == 0 && tid == 0 && bad) flag[0] = 1;
#pragma unroll
  for (int q = 0; q < 16; ++q) Dr[rqs + 4 * q][col] = aT[q];
  __syncthreads();
  const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32, li = lane & 15, lk = lane >> 4;
  d4v acc[2][2];
  if (lpart) {
    mma64<true>(Or, &Dr[0][0], acc, wi, wj, li, lk);  // A_ik D_k^T
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) C[(wi + 16 * a + lk + 4 * r) * Np + wj + 16 * b + li] = acc[a][b][r];
    return;
  }
  mma64<false>(Dr, &Ok[0][0], acc, wi, wj, li, lk);  // D_k B_kj
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) Or[wi + 16 * a + lk + 4 * r][wj + 16 * b + li] = acc[a][b][r];
  __syncthreads();
  for (int e = tid; e < kHb * kHb / 2; e += 256) {
    const int r = e >> 5, m = (e & 31) * 2;
    *reinterpret_cast<d2v*>(C + r * Np + m) = *reinterpret_cast<const d2v*>(&Or[r][m]);
  }
  if (tid < kHb) {
    double sq = 0.0;
    for (int r = 0; r < kHb; ++r) sq += Or[r][tid] * Or[r][tid];
    colsq[(g - nbelow) * kHb + tid] += sq;
  }
}

// Step 3.  Workgroups below ntri: the lower-triangle tiles (a >= b) of the trailing matrix,
// A_ij -= L_ik L_jk^T with i = k + 1 + a, j = k + 1 + b.  The others: B_ij -= L_ik T_kj for
// i = k + 1 + a, j <= k.
__global__ __launch_bounds__(256) void hinv_update_kernel(double* __restrict__ A, double* __restrict__ B, int64_t Np,
                                                          int64_t k, int64_t ntri) {
  __shared__ double Ar[kHb][kHr];
  __shared__ double Bs[kHb * kHs];  // rows of L_jk (stride kHr) or T_kj k-major (stride kHs)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32, li = lane & 15, lk = lane >> 4;
  const int64_t g = blockIdx.x, kb = k * kHb;
  double* C;
  d4v acc[2][2];
  if (g < ntri) {
    // g = a (a + 1) / 2 + b, 0 <= b <= a
    int64_t a = static_cast<int64_t>((sqrt(8.0 * static_cast<double>(g) + 1.0) - 1.0) * 0.5);
    while (a * (a + 1) / 2 > g) --a;
    while ((a + 1) * (a + 2) / 2 <= g) ++a;
    const int64_t b = g - a * (a + 1) / 2;
    const int64_t ib = (k + 1 + a) * kHb, jb = (k + 1 + b) * kHb;
    load_rows(Ar, A + ib * Np + kb, Np, tid);
    load_rows(reinterpret_cast<double(*)[kHr]>(Bs), A + jb * Np + kb, Np, tid);
    C = A + ib * Np + jb;
  } else {
    const int64_t h = g - ntri, a = h / (k + 1), j = h - a * (k + 1);
    const int64_t ib = (k + 1 + a) * kHb, jb = j * kHb;
    load_rows(Ar, A + ib * Np + kb, Np, tid);
    load_kmaj(reinterpret_cast<double(*)[kHs]>(Bs), B + kb * Np + jb, Np, tid);
    C = B + ib * Np + jb;
  }
  // this lane's elements of the output tile, read while the products run
  double old[2][2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) old[a][b][r] = C[(wi + 16 * a + lk + 4 * r) * Np + wj + 16 * b + li];
  __syncthreads();
  if (g < ntri)
    mma64<true>(Ar, Bs, acc, wi, wj, li, lk);
  else
    mma64<false>(Ar, Bs, acc, wi, wj, li, lk);
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) C[(wi + 16 * a + lk + 4 * r) * Np + wj + 16 * b + li] = old[a][b][r] - acc[a][b][r];
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
    const int64_t nbelow = nblk - 1 - k;
    hipLaunchKernelGGL(hinv_step_kernel, dim3(static_cast<unsigned>(nbelow + k + 1)), dim3(256), 0, stream, w.A, w.B,
                       Np, k, nbelow, w.colsq, w.flag);
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
